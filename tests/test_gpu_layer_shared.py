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


def _needles_kept(x, budget, idx):
    """Needles of the groups that have SRHs (and the sinks) win their pooling
    neighbourhoods in the layer score; all of them are kept when the prefix
    budget covers every such neighbourhood."""
    w = x.workload
    G = w.n_q_heads // w.n_kv_heads
    groups = [g for g in range(w.n_kv_heads) if x.srh_mask[g * G:(g + 1) * G].any()]
    if budget - w.window < (len(groups) * w.n_needle + w.n_sink) * w.pool_kernel:
        return False
    for (b, g), pos in x.needles.items():
        if g in groups:
            assert set(pos.tolist()) <= set(idx[b, 0].tolist()), (b, g)
    return True


def _paper_stack(xs, budgets, gpu):
    dts = [H.device_tensors(x, gpu) for x in xs]
    q, k, v = [d[0] for d in dts], [d[1] for d in dts], [d[2] for d in dts]
    masks = np.stack([x.srh_mask for x in xs])
    ps = [_problem(xs[l], q[l], k[l], v[l], dts[0][3]) for l in range(len(xs))]
    idxs, kos, vos, scores = C.compress_layers(ps[0], q, k, v, masks, budgets, want_scores=True)
    ref = [C.compress_layer(ps[l], q[l], k[l], v[l], masks[l], int(budgets[l]), want_scores=True)
           for l in range(len(xs))]
    torch.cuda.synchronize()
    for l in range(len(xs)):
        for got, want in zip((idxs[l], kos[l], vos[l], scores[l]), ref[l]):
            assert torch.equal(got, want), f"layer {l} differs from the per-layer call"
    return idxs, kos, vos, scores


def test_paper_setting_stack(gpu):
    """The paper's own setting (section 4): W = 8, max pooling 5, the top 4
    SRHs of each layer, the layer-shared index set and budgets within
    [32, 3 x 512], at L = 9001 over 6 layers with the full stack's first
    budgets: one multi-layer call, bit-identical to per-layer calls, every
    layer against the oracle."""
    w = wl.get("paper", seq_len=9001, n_layers=6)
    budgets = [int(b) for b in wl.layer_budgets(wl.get("paper"))[:6]]
    xs = [wl.make_layer(w, l, seed=41, budget=B) for l, B in enumerate(budgets)]
    _say(f"case paper setting stack, budgets {budgets}, SRH masks "
         f"{[np.flatnonzero(x.srh_mask).tolist() for x in xs]}")
    idxs, kos, vos, scores = _paper_stack(xs, budgets, gpu)
    kept_all = 0
    for l, x in enumerate(xs):
        idx = idxs[l].cpu().numpy()
        swaps = _check(x, budgets[l], scores[l].cpu().numpy(), idx, H.raw_bits(kos[l]),
                       H.raw_bits(vos[l]))
        kept_all += _needles_kept(x, budgets[l], idx)
        _say(f"  layer {l} ok, boundary swaps {swaps}")
    assert kept_all > 0


def test_paper_setting_full_stack(gpu):
    """The same setting at the benchmark's size: 32 layers at L = 32768,
    inputs drawn on the device; one multi-layer call, bit-identical to
    per-layer calls on every layer, and three layers against the oracle."""
    w = wl.get("paper")
    layers = [wl.make_layer_device(w, l, 0, gpu) for l in range(w.n_layers)]
    budgets = [d["budget"] for d in layers]
    _say(f"case paper setting full stack, budgets {budgets}")
    q = [d["q_win"] for d in layers]
    k = [d["k"] for d in layers]
    v = [d["v"] for d in layers]
    cu, cu_host = layers[0]["cu_seqlens"], layers[0]["cu_seqlens_host"]
    masks = np.stack([d["srh_mask"] for d in layers])
    ps = [C.Problem(q[l], k[l], v[l], cu, cu_seqlens_host=cu_host, pool_kernel=w.pool_kernel,
                    pool_type=w.pool_type, index_mode=C.INDEX_LAYER) for l in range(w.n_layers)]
    idxs, kos, vos, scores = C.compress_layers(ps[0], q, k, v, masks, budgets, want_scores=True)
    torch.cuda.synchronize()
    for l in range(w.n_layers):
        ref = C.compress_layer(ps[l], q[l], k[l], v[l], masks[l], budgets[l], want_scores=True)
        torch.cuda.synchronize()
        for got, want in zip((idxs[l], kos[l], vos[l], scores[l]), ref):
            assert torch.equal(got, want), f"layer {l} differs from the per-layer call"
        del ref
    for l in (0, 13, 31):
        d = layers[l]
        x = wl.LayerInputs(workload=w, layer=l, cu_seqlens=cu_host, srh_mask=d["srh_mask"],
                           budget=d["budget"], q_win=d["q_win"].float().cpu().numpy(),
                           k=d["k"].float().cpu().numpy(), v=d["v"].float().cpu().numpy(),
                           needles=d["needles"])
        idx = idxs[l].cpu().numpy()
        swaps = _check(x, budgets[l], scores[l].cpu().numpy(), idx, H.raw_bits(kos[l]),
                       H.raw_bits(vos[l]))
        _needles_kept(x, budgets[l], idx)
        _say(f"  layer {l} matches the oracle, boundary swaps {swaps}")
