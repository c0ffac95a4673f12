"""GPU parity of the multi-layer entry points (compresskv_compress_layers,
compresskv_score_layers): every layer against the fp64 oracle under the rules
of tests/parity_helpers.py, and bit-identity with per-layer calls."""
import sys

import numpy as np
import pytest
import torch

from paper_2606_24467_amd import compresskv as C
from paper_2606_24467_amd import workloads as wl
from tests import parity_helpers as H

pytestmark = pytest.mark.gpu


PATHS = {"two": C.SCORE_TWO_PASS, "one": C.SCORE_ONE_PASS}


@pytest.fixture(autouse=True, params=sorted(PATHS))
def scoring_path(request, monkeypatch):
    """Every case runs on the two-pass path (the library's own choice) and on
    the single pass (skipped, with the library's reason, where it does not
    apply to some layer); the per-layer calls it is compared with use the
    same scoring field."""
    monkeypatch.setattr(H, "SCORING", PATHS[request.param])
    return request.param


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


def _problem(q, k, v, cu, cu_host, w, masks=None):
    return H.problem(q, k, v, cu, masks=masks, cu_seqlens_host=cu_host,
                     pool_kernel=w.pool_kernel, pool_type=w.pool_type)


def _host_inputs(w, layer, d) -> wl.LayerInputs:
    """A device-generated layer as oracle inputs (the values the kernels read)."""
    return wl.LayerInputs(workload=w, layer=layer, cu_seqlens=d["cu_seqlens_host"],
                          srh_mask=d["srh_mask"], budget=d["budget"],
                          q_win=d["q_win"].float().cpu().numpy(),
                          k=d["k"].float().cpu().numpy(), v=d["v"].float().cpu().numpy(),
                          needles=d["needles"])


def _check_layer(x, budget, scores, idx, k_out, v_out):
    ora = H.run_oracle(x, budget)
    W = x.workload.window
    H.check_scores(scores, ora, x.cu_seqlens, W)
    swaps = H.check_indices(idx, ora, x.cu_seqlens, W, budget)
    H.check_gather(k_out, v_out, idx, x.bits("k"), x.bits("v"), x.cu_seqlens)
    return swaps


def _check_needles(x, budget, idx):
    """Needles (and sinks) win their pooling neighbourhoods; all of them are
    kept when the prefix budget covers every such neighbourhood."""
    w = x.workload
    if budget - w.window < (w.n_needle + w.n_sink) * w.pool_kernel:
        return
    for (b, g), pos in x.needles.items():
        assert set(pos.tolist()) <= set(idx[b, g].tolist()), (b, g)


def _per_layer(p, q, k, v, masks, budgets):
    out = []
    for l in range(len(k)):
        out.append(C.compress_layer(p[l], q[l], k[l], v[l], masks[l], int(budgets[l]),
                                    want_scores=True))
    return out


def test_compress_layers_matches_oracle_ragged(gpu):
    w = wl.get("ragged8", batch=3, n_layers=5, ragged=(700, 2600), srh_per_group=(1, 3),
               n_needle=4)
    budgets = [64, 300, 2600, 32, 1111]     # 2600 >= every length (all kept); 32 = W
    xs = [wl.make_layer(w, l, seed=21, budget=B) for l, B in enumerate(budgets)]
    _say(f"case ragged stack L={np.diff(xs[0].cu_seqlens).tolist()} budgets={budgets}")
    dts = [H.device_tensors(x, gpu) for x in xs]
    q, k, v = [d[0] for d in dts], [d[1] for d in dts], [d[2] for d in dts]
    cu = dts[0][3]
    masks = np.stack([x.srh_mask for x in xs])
    ps = [_problem(q[l], k[l], v[l], cu, xs[0].cu_seqlens, w, masks) for l in range(w.n_layers)]
    idxs, kos, vos, scores = C.compress_layers(ps[0], q, k, v, masks, budgets, want_scores=True)
    ref = _per_layer(ps, q, k, v, masks, budgets)
    only_scores = C.score_layers(ps[0], q, k, masks)
    torch.cuda.synchronize()
    for l, x in enumerate(xs):
        for got, want in zip((idxs[l], kos[l], vos[l], scores[l]), ref[l]):
            assert torch.equal(got, want), f"layer {l} differs from the per-layer call"
        assert torch.equal(only_scores[l], scores[l])
        swaps = _check_layer(x, budgets[l], scores[l].cpu().numpy(), idxs[l].cpu().numpy(),
                             H.raw_bits(kos[l]), H.raw_bits(vos[l]))
        _say(f"  layer {l} ok, boundary swaps {swaps}")


def test_compress_layers_qwen_shape_reduced(gpu):
    w = wl.get("qwen128k", seq_len=12000 + 5, n_layers=3, n_needle=8)
    budgets = [200, 64, 1777]
    xs = [wl.make_layer(w, l, seed=22, budget=B) for l, B in enumerate(budgets)]
    _say(f"case qwen stack L={w.seq_len} budgets={budgets}")
    dts = [H.device_tensors(x, gpu) for x in xs]
    q, k, v = [d[0] for d in dts], [d[1] for d in dts], [d[2] for d in dts]
    masks = np.stack([x.srh_mask for x in xs])
    p = _problem(q[0], k[0], v[0], dts[0][3], xs[0].cu_seqlens, w, masks)
    idxs, kos, vos, scores = C.compress_layers(p, q, k, v, masks, budgets, want_scores=True)
    torch.cuda.synchronize()
    for l, x in enumerate(xs):
        _check_layer(x, budgets[l], scores[l].cpu().numpy(), idxs[l].cpu().numpy(),
                     H.raw_bits(kos[l]), H.raw_bits(vos[l]))
        _check_needles(x, budgets[l], idxs[l].cpu().numpy())


def test_full_32_layer_stack(gpu, scoring_path):
    """The 32-layer Llama-3-8B-shaped stack at L = 32768 as the benchmark runs
    it: one multi-layer call, bit-identical to per-layer calls on every layer,
    and checked against the oracle in full: every layer on the two-pass path
    (the library's own choice, the benchmarked one), two sampled layers on
    the single pass."""
    w = wl.get("llama32")
    layers = [wl.make_layer_device(w, l, 0, gpu) for l in range(w.n_layers)]
    _say(f"case llama32 full stack, budgets {[d['budget'] for d in layers]}")
    q = [d["q_win"] for d in layers]
    k = [d["k"] for d in layers]
    v = [d["v"] for d in layers]
    cu, cu_host = layers[0]["cu_seqlens"], layers[0]["cu_seqlens_host"]
    masks = np.stack([d["srh_mask"] for d in layers])
    ps = [_problem(q[l], k[l], v[l], cu, cu_host, w, masks) for l in range(w.n_layers)]
    budgets = [d["budget"] for d in layers]
    idxs, kos, vos, scores = C.compress_layers(ps[0], q, k, v, masks, budgets, want_scores=True)
    ref = _per_layer(ps, q, k, v, masks, budgets)
    torch.cuda.synchronize()
    for l in range(w.n_layers):
        for got, want in zip((idxs[l], kos[l], vos[l], scores[l]), ref[l]):
            assert torch.equal(got, want), f"layer {l} differs from the per-layer call"
    del ref
    for l in (range(w.n_layers) if scoring_path == "two" else (0, 17)):
        x = _host_inputs(w, l, layers[l])
        swaps = _check_layer(x, budgets[l], scores[l].cpu().numpy(), idxs[l].cpu().numpy(),
                             H.raw_bits(kos[l]), H.raw_bits(vos[l]))
        _check_needles(x, budgets[l], idxs[l].cpu().numpy())
        _say(f"  layer {l} matches the oracle, boundary swaps {swaps}")


@pytest.mark.parametrize("name,sampled", [("qwen128k", (0, 19)), ("ragged8", (0, 23))])
def test_full_stack_other_shapes(gpu, scoring_path, name, sampled):
    """The Qwen-shaped stack (28 layers, 28q/4kv heads, L = 131072, W = 64,
    Dirichlet budgets) and the ragged batch (32 layers, 8 sequences of
    4096-16384 tokens) at full size: one multi-layer call, bit-identical to
    per-layer calls on every layer, and sampled layers against the oracle in
    full."""
    w = wl.get(name)
    layers = [wl.make_layer_device(w, l, 0, gpu) for l in range(w.n_layers)]
    _say(f"case {name} full stack, lengths {np.diff(layers[0]['cu_seqlens_host']).tolist()}, "
         f"budgets {[d['budget'] for d in layers]}")
    q = [d["q_win"] for d in layers]
    k = [d["k"] for d in layers]
    v = [d["v"] for d in layers]
    cu, cu_host = layers[0]["cu_seqlens"], layers[0]["cu_seqlens_host"]
    masks = np.stack([d["srh_mask"] for d in layers])
    ps = [_problem(q[l], k[l], v[l], cu, cu_host, w, masks) for l in range(w.n_layers)]
    budgets = [d["budget"] for d in layers]
    idxs, kos, vos, scores = C.compress_layers(ps[0], q, k, v, masks, budgets, want_scores=True)
    ref = _per_layer(ps, q, k, v, masks, budgets)
    torch.cuda.synchronize()
    for l in range(w.n_layers):
        for got, want in zip((idxs[l], kos[l], vos[l], scores[l]), ref[l]):
            assert torch.equal(got, want), f"layer {l} differs from the per-layer call"
    del ref
    for l in sampled:
        x = _host_inputs(w, l, layers[l])
        swaps = _check_layer(x, budgets[l], scores[l].cpu().numpy(), idxs[l].cpu().numpy(),
                             H.raw_bits(kos[l]), H.raw_bits(vos[l]))
        _check_needles(x, budgets[l], idxs[l].cpu().numpy())
        _say(f"  layer {l} matches the oracle, boundary swaps {swaps}")


def test_many_layers_short_sequences(gpu, scoring_path):
    """32 layers x 8 sequences of 2000-3000 tokens: enough units for
    several chunks per workgroup, but fewer chunks per sequence than the
    one-chunk tail, so every chunk goes one per workgroup in its own order;
    bit-identical to per-layer calls, two layers against the oracle."""
    w = wl.get("ragged8", ragged=(2000, 3000), n_needle=4)
    layers = [wl.make_layer_device(w, l, 0, gpu) for l in range(w.n_layers)]
    _say(f"case many short sequences, lengths {np.diff(layers[0]['cu_seqlens_host']).tolist()}")
    q = [d["q_win"] for d in layers]
    k = [d["k"] for d in layers]
    v = [d["v"] for d in layers]
    cu, cu_host = layers[0]["cu_seqlens"], layers[0]["cu_seqlens_host"]
    masks = np.stack([d["srh_mask"] for d in layers])
    ps = [_problem(q[l], k[l], v[l], cu, cu_host, w, masks) for l in range(w.n_layers)]
    budgets = [d["budget"] for d in layers]
    idxs, kos, vos, scores = C.compress_layers(ps[0], q, k, v, masks, budgets, want_scores=True)
    ref = _per_layer(ps, q, k, v, masks, budgets)
    torch.cuda.synchronize()
    for l in range(w.n_layers):
        for got, want in zip((idxs[l], kos[l], vos[l], scores[l]), ref[l]):
            assert torch.equal(got, want), f"layer {l} differs from the per-layer call"
    del ref
    for l in (0, 31):
        x = _host_inputs(w, l, layers[l])
        swaps = _check_layer(x, budgets[l], scores[l].cpu().numpy(), idxs[l].cpu().numpy(),
                             H.raw_bits(kos[l]), H.raw_bits(vos[l]))
        _say(f"  layer {l} matches the oracle, boundary swaps {swaps}")
