"""Two passes in one launch (CKV_SCORE_TWO_PASS on bf16 inputs with at most 8
row tiles per group; CKV_SCORE_AUTO where the sequences are also long) against the same passes in two launches
(CKV_SCORE_TWO_LAUNCHES): the normalisers merge the same partials in the same
order, so every output must agree bit for bit, whatever the wait bound of
the in-launch exchange (default, no waiting, everything left to the catch-up
kernel).  The oracle check of the one-launch results is in the other GPU
tests, which run the library's default path; here one case is also checked
against the oracle directly."""
import sys

import numpy as np
import pytest
import torch

from paper_2606_24467_amd import compresskv as C
from paper_2606_24467_amd import workloads as wl
from tests import parity_helpers as H

pytestmark = pytest.mark.gpu

SPINS = (C.SPIN_DEFAULT, 0, C.SPIN_CATCHUP_ALL)


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


def _layer_outputs(x, dev, scoring, spin, budget):
    q, k, v, cu = H.device_tensors(x, dev)
    p = H.problem(q, k, v, cu, masks=x.srh_mask, cu_seqlens_host=x.cu_seqlens,
                  scoring=scoring, spin_limit=spin, pool_kernel=x.workload.pool_kernel,
                  pool_type=x.workload.pool_type,
                  index_mode=C.INDEX_LAYER if x.workload.index_layer else C.INDEX_PER_GROUP)
    path = C.compresskv_scoring_path(p, x.srh_mask)
    out = C.compress_layer(p, q, k, v, x.srh_mask, budget, want_scores=True)
    torch.cuda.synchronize()
    return path, [t.clone() for t in out]


CASES = [
    # name, workload overrides, budget
    ("llama 8k, 1-3 SRHs per group", "llama1", dict(seq_len=8192 + 7, n_needle=8,
                                                     srh_per_group=(1, 3)), 600),
    ("ragged batch of 5", "ragged8", dict(batch=5, ragged=(1100, 9000), n_needle=4), 400),
    ("head dim 64", "llama1", dict(seq_len=5000, head_dim=64, n_needle=4), 256),
    ("window 8, pooling 5, layer-shared", "paper", dict(seq_len=6000, n_layers=1), 300),
    ("window 48, 2 SRHs (6 row tiles)", "llama1", dict(seq_len=40000, window=48, n_needle=8,
                                                         srh_per_group=(2,)), 2000),
    ("Qwen shape, window 64, 2 SRHs (8 row tiles)", "qwen128k", dict(seq_len=20000 + 3,
                                                                    n_layers=1, n_needle=8),
     900),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_one_launch_matches_two_launches_bitwise(gpu, case):
    _, name, kw, budget = case
    w = wl.get(name, **kw)
    x = wl.make_layer(w, 0, seed=31)
    _say(f"case {case[0]}: L={np.diff(x.cu_seqlens).tolist()[:8]} budget={budget}")
    path, ref = _layer_outputs(x, gpu, C.SCORE_TWO_LAUNCHES, C.SPIN_DEFAULT, budget)
    assert path == 2
    for spin in SPINS:
        path, got = _layer_outputs(x, gpu, C.SCORE_TWO_PASS, spin, budget)
        assert path == 3, "bf16 with at most 8 row tiles runs in one launch"
        for a, b, what in zip(got, ref, ("idx", "k_out", "v_out", "scores")):
            assert torch.equal(a, b), f"{what} differs (spin_limit {spin})"
    _say("  ok")


def test_one_launch_matches_oracle(gpu):
    w = wl.get("ragged8", batch=3, ragged=(3000, 12000), n_needle=6)
    x = wl.make_layer(w, 0, seed=32)
    path, (idx, k_out, v_out, scores) = _layer_outputs(x, gpu, C.SCORE_TWO_PASS,
                                                       C.SPIN_DEFAULT, 700)
    assert path == 3
    ora = H.run_oracle(x, 700)
    H.check_scores(scores.cpu().numpy(), ora, x.cu_seqlens, w.window)
    H.check_indices(idx.cpu().numpy(), ora, x.cu_seqlens, w.window, 700)
    H.check_gather(H.raw_bits(k_out), H.raw_bits(v_out), idx.cpu().numpy(), x.bits("k"),
                   x.bits("v"), x.cu_seqlens)


def test_multi_layer_one_launch_matches_two_launches(gpu):
    """A multi-layer call (layers with 1-3 SRHs per group, ragged batch) in
    one launch against two launches, and against per-layer calls."""
    w = wl.get("ragged8", batch=3, n_layers=6, ragged=(2000, 11000), srh_per_group=(1, 3),
               n_needle=4)
    budgets = [128, 500, 3000, 64, 999, 32]
    xs = [wl.make_layer(w, l, seed=33, budget=B) for l, B in enumerate(budgets)]
    dts = [H.device_tensors(x, gpu) for x in xs]
    q, k, v = [d[0] for d in dts], [d[1] for d in dts], [d[2] for d in dts]
    cu = dts[0][3]
    masks = np.stack([x.srh_mask for x in xs])
    outs = {}
    for scoring, spin in ((C.SCORE_TWO_LAUNCHES, C.SPIN_DEFAULT),
                          (C.SCORE_TWO_PASS, C.SPIN_DEFAULT), (C.SCORE_TWO_PASS, 0),
                          (C.SCORE_TWO_PASS, C.SPIN_CATCHUP_ALL)):
        p = H.problem(q[0], k[0], v[0], cu, masks=masks, cu_seqlens_host=xs[0].cu_seqlens,
                      scoring=scoring, spin_limit=spin)
        res = C.compress_layers(p, q, k, v, masks, budgets, want_scores=True)
        torch.cuda.synchronize()
        outs[(scoring, spin)] = res
    ref = outs[(C.SCORE_TWO_LAUNCHES, C.SPIN_DEFAULT)]
    for key, res in outs.items():
        for l in range(w.n_layers):
            for part in range(4):
                assert torch.equal(res[part][l], ref[part][l]), (key, l, part)
    for l in (0, 2):
        pl_ = H.problem(q[l], k[l], v[l], cu, masks=masks[l], cu_seqlens_host=xs[0].cu_seqlens,
                        scoring=C.SCORE_TWO_PASS)
        one = C.compress_layer(pl_, q[l], k[l], v[l], masks[l], budgets[l], want_scores=True)
        torch.cuda.synchronize()
        for part in range(4):
            assert torch.equal(one[part], ref[part][l]), (l, part)


def test_full_stack_repeated_calls_match_two_launches(gpu):
    """The benchmark's 32-layer stack (L = 32768, inputs drawn on the device):
    ten one-launch calls in a row, each bit for bit equal to the two-launch
    call, so no call's result depends on how its exchange was timed."""
    w = wl.get("llama32")
    layers = [wl.make_layer_device(w, l, 0, gpu) for l in range(w.n_layers)]
    q = [d["q_win"] for d in layers]
    k = [d["k"] for d in layers]
    masks = np.stack([d["srh_mask"] for d in layers])
    cu, cu_host = layers[0]["cu_seqlens"], layers[0]["cu_seqlens_host"]
    probs = {s: C.Problem(q[0], k[0], layers[0]["v"], cu, cu_seqlens_host=cu_host,
                          pool_kernel=w.pool_kernel, pool_type=w.pool_type, scoring=s)
             for s in (C.SCORE_AUTO, C.SCORE_TWO_LAUNCHES)}
    assert C.compresskv_scoring_path(probs[C.SCORE_AUTO], masks[0]) == 3
    ref = C.score_layers(probs[C.SCORE_TWO_LAUNCHES], q, k, masks)
    p = probs[C.SCORE_AUTO]
    ws = C.layers_workspace(p, masks, gpu)
    out = torch.empty_like(ref)
    for call in range(10):
        out.fill_(float("nan"))
        C.compresskv_score_layers(p, q, k, masks, out, ws, torch.cuda.current_stream())
        torch.cuda.synchronize()
        assert torch.equal(out, ref), f"call {call} differs from the two launches"
    _say("  10 calls equal")
