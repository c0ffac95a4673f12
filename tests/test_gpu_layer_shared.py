"""GPU parity of the layer-shared index set (section 3.3: one selection per
sequence from all of the layer's SRHs, kept by every KV group) against the
fp64 oracle in its LAYER_SHARED mode, under the rules of
tests/parity_helpers.py.  Groups without an SRH are part of every case."""
import sys

import numpy as np
import pytest
import torch

import oracle as O
from paper_2606_24467_amd import compresskv as C
from paper_2606_24467_amd import workloads as wl
from tests import parity_helpers as H

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


@pytest.fixture(autouse=True)
def _two_pass(monkeypatch):
    monkeypatch.delenv("CKV_PATH", raising=False)


def _drop_groups(x: wl.LayerInputs, groups):
    """Remove every SRH of the given KV groups (the layer keeps the others)."""
    G = x.srh_mask.shape[0] // x.workload.n_kv_heads
    for g in groups:
        x.srh_mask[g * G:(g + 1) * G] = 0
    return x


def _problem(x, q, k, v, cu):
    w = x.workload
    return C.Problem(q, k, v, cu, cu_seqlens_host=x.cu_seqlens, pool_kernel=w.pool_kernel,
                     pool_type=w.pool_type, index_mode=C.INDEX_LAYER)


def _check(x, budget, scores, idx, k_out, v_out):
    ora = H.run_oracle(x, budget, index_mode=O.LAYER_SHARED)
    W = x.workload.window
    H.check_scores(scores, ora, x.cu_seqlens, W)
    swaps = H.check_indices(idx, ora, x.cu_seqlens, W, budget)
    kb = x.bits("k") if x.dtype == wl.BF16 else x.k.view(np.uint32)
    vb = x.bits("v") if x.dtype == wl.BF16 else x.v.view(np.uint32)
    H.check_gather(k_out, v_out, idx, kb, vb, x.cu_seqlens)
    # one index set per sequence: every group's row is the same
    assert np.all(idx == idx[:, :1]), "groups hold different index sets"
    assert np.all(scores[:, :] == scores[:1, :]), "groups hold different layer scores"
    return swaps


@pytest.mark.parametrize("budget", [32, 150, 700])
def test_layer_set_ragged_batch(gpu, budget):
    w = wl.get("ragged8", batch=4, ragged=(400, 1800), srh_per_group=(1, 3), n_needle=4)
    x = _drop_groups(wl.make_layer(w, 0, seed=31, budget=budget), [1, 4, 5])
    _say(f"case layer set ragged L={np.diff(x.cu_seqlens).tolist()} budget={budget} "
         f"mask={x.srh_mask.tolist()}")
    q, k, v, cu = H.device_tensors(x, gpu)
    p = _problem(x, q, k, v, cu)
    idx, k_out, v_out, scores = C.compress_layer(p, q, k, v, x.srh_mask, budget,
                                                 want_scores=True)
    torch.cuda.synchronize()
    swaps = _check(x, budget, scores.cpu().numpy(), idx.cpu().numpy(), H.raw_bits(k_out),
                   H.raw_bits(v_out))
    _say(f"  ok, boundary swaps {swaps}")


def test_layer_set_single_srh_in_the_layer(gpu):
    w = wl.get("tiny", seq_len=900)
    x = wl.make_layer(w, 0, seed=32, budget=100)
    x.srh_mask[:] = 0
    x.srh_mask[x.srh_mask.shape[0] - 1] = 1        # one SRH, in the last group
    _say(f"case layer set one SRH L={np.diff(x.cu_seqlens).tolist()} mask={x.srh_mask.tolist()}")
    q, k, v, cu = H.device_tensors(x, gpu)
    p = _problem(x, q, k, v, cu)
    idx, k_out, v_out, scores = C.compress_layer(p, q, k, v, x.srh_mask, 100, want_scores=True)
    torch.cuda.synchronize()
    _check(x, 100, scores.cpu().numpy(), idx.cpu().numpy(), H.raw_bits(k_out),
           H.raw_bits(v_out))


def test_layer_set_score_then_select_entry_points(gpu):
    """compresskv_score writes the layer score into every row; compresskv_select
    reads row 0 and writes the one index set into every group's row."""
    w = wl.get("llama32", seq_len=5000 + 3, n_layers=1, n_needle=8)
    x = _drop_groups(wl.make_layer(w, 0, seed=33, budget=600), [0, 7])
    _say(f"case layer set score+select L={np.diff(x.cu_seqlens).tolist()}")
    q, k, v, cu = H.device_tensors(x, gpu)
    p = _problem(x, q, k, v, cu)
    scores = C.score(p, q, k, x.srh_mask)
    idx = C.select(p, scores, 600)
    k_out, v_out = C.gather(p, k, v, idx, 600)
    ref = C.compress_layer(p, q, k, v, x.srh_mask, 600, want_scores=True)
    torch.cuda.synchronize()
    for got, want in zip((idx, k_out, v_out, scores), ref):
        assert torch.equal(got, want)
    _check(x, 600, scores.cpu().numpy(), idx.cpu().numpy(), H.raw_bits(k_out),
           H.raw_bits(v_out))


def test_layer_set_multi_layer_call(gpu):
    """compresskv_compress_layers with the layer-shared set: bit-identical to
    per-layer calls, and every layer against the oracle."""
    w = wl.get("ragged8", batch=3, n_layers=4, ragged=(600, 2100), srh_per_group=(1, 2),
               n_needle=4)
    budgets = [64, 400, 2100, 32]
    drops = [[], [2, 3], [0, 1, 2, 3, 4, 5, 6], [5]]
    xs = [_drop_groups(wl.make_layer(w, l, seed=34, budget=B), drops[l])
          for l, B in enumerate(budgets)]
    _say(f"case layer set stack L={np.diff(xs[0].cu_seqlens).tolist()} budgets={budgets}")
    dts = [H.device_tensors(x, gpu) for x in xs]
    q, k, v = [d[0] for d in dts], [d[1] for d in dts], [d[2] for d in dts]
    cu = dts[0][3]
    ps = [_problem(xs[l], q[l], k[l], v[l], cu) for l in range(w.n_layers)]
    masks = np.stack([x.srh_mask for x in xs])
    idxs, kos, vos, scores = C.compress_layers(ps[0], q, k, v, masks, budgets, want_scores=True)
    only_scores = C.score_layers(ps[0], q, k, masks)
    ref = [C.compress_layer(ps[l], q[l], k[l], v[l], masks[l], budgets[l], want_scores=True)
           for l in range(w.n_layers)]
    torch.cuda.synchronize()
    for l, x in enumerate(xs):
        for got, want in zip((idxs[l], kos[l], vos[l], scores[l]), ref[l]):
            assert torch.equal(got, want), f"layer {l} differs from the per-layer call"
        assert torch.equal(only_scores[l], scores[l])
        swaps = _check(x, budgets[l], scores[l].cpu().numpy(), idxs[l].cpu().numpy(),
                       H.raw_bits(kos[l]), H.raw_bits(vos[l]))
        _say(f"  layer {l} ok, boundary swaps {swaps}")
