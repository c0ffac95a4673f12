"""HIP graphs: the eviction path makes no allocation, memset or copy, so a
caller can capture it.  Each case captures the C-ABI call once, replays the
graph several times with eager work and synchronisations between the
replays, and checks every replay bit for bit against the eager call on the
same inputs (the kernels are deterministic); the outputs are overwritten
before each replay so a replay that skips a write is caught.  A last replay
after the inputs changed in place must follow the new inputs."""
import sys

import numpy as np
import pytest
import torch

from paper_2606_24467_amd import compresskv as C
from paper_2606_24467_amd import workloads as wl

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


def _poison(outs):
    for t in outs:
        if t.dtype == torch.int32:
            t.fill_(-7)
        else:
            t.fill_(float("nan"))


def _other_eager_work(gpu):
    x = torch.randn((1 << 20,), device=gpu)
    assert torch.isfinite(x.sum()).item()
    torch.cuda.synchronize()


def _replays_match(g, outs, ref, gpu, n=3):
    for r in range(n):
        _poison(outs)
        _other_eager_work(gpu)
        g.replay()
        torch.cuda.synchronize()
        for i, (got, want) in enumerate(zip(outs, ref)):
            assert torch.equal(got, want), f"replay {r}: output {i} differs from the eager call"


SCORING = {"auto": C.SCORE_AUTO, "one launch": C.SCORE_TWO_PASS,
           "two launches": C.SCORE_TWO_LAUNCHES}


@pytest.mark.parametrize("scoring", sorted(SCORING))
def test_multi_layer_call_in_a_graph(gpu, scoring):
    w = wl.get("llama32", seq_len=5000 + 7, n_layers=3)
    layers = [wl.make_layer_device(w, l, 0, gpu) for l in range(w.n_layers)]
    q = [d["q_win"] for d in layers]
    k = [d["k"] for d in layers]
    v = [d["v"] for d in layers]
    masks = np.stack([d["srh_mask"] for d in layers])
    budgets = [d["budget"] for d in layers]
    _say(f"case graph, 3-layer stack L={w.seq_len} budgets {budgets}, scoring {scoring}")
    p = C.Problem(q[0], k[0], v[0], layers[0]["cu_seqlens"],
                  cu_seqlens_host=layers[0]["cu_seqlens_host"], pool_kernel=w.pool_kernel,
                  pool_type=w.pool_type, scoring=SCORING[scoring])
    idxs = [torch.empty((1, w.n_kv_heads, B), dtype=torch.int32, device=gpu) for B in budgets]
    k_outs = [torch.empty((1, w.n_kv_heads, B, w.head_dim), dtype=k[0].dtype, device=gpu)
              for B in budgets]
    v_outs = [torch.empty_like(t) for t in k_outs]
    scores = torch.empty((w.n_layers, w.n_kv_heads, p.total_tokens), dtype=torch.float32,
                         device=gpu)
    ws = C.layers_workspace(p, masks, gpu)
    call = C.LayersCall(p, q, k, v, masks, budgets, idxs, k_outs, v_outs, scores, ws)
    outs = idxs + k_outs + v_outs + [scores]

    call()
    torch.cuda.synchronize()
    ref = [t.clone() for t in outs]
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call()
    torch.cuda.synchronize()
    _replays_match(g, outs, ref, gpu)

    # new keys in layer 1: the replay reads the live buffers
    k[1].copy_(torch.randn(k[1].shape, device=gpu).to(k[1].dtype))
    call()
    torch.cuda.synchronize()
    ref2 = [t.clone() for t in outs]
    assert not torch.equal(ref2[1], ref[1])
    _replays_match(g, outs, ref2, gpu, n=2)


@pytest.mark.parametrize("scoring", sorted(SCORING))
def test_single_layer_call_in_a_graph(gpu, scoring):
    w = wl.get("llama1", seq_len=3000 + 3, n_needle=4, batch=2, ragged=(1500, 3003))
    d = wl.make_layer_device(w, 0, 0, gpu)
    B = 300
    _say(f"case graph, single layer lengths {np.diff(d['cu_seqlens_host']).tolist()} budget {B}, "
         f"scoring {scoring}")
    p = C.Problem(d["q_win"], d["k"], d["v"], d["cu_seqlens"],
                  cu_seqlens_host=d["cu_seqlens_host"], pool_kernel=w.pool_kernel,
                  pool_type=w.pool_type, scoring=SCORING[scoring])
    shape = (w.batch, w.n_kv_heads, B, w.head_dim)
    idx = torch.empty(shape[:3], dtype=torch.int32, device=gpu)
    k_out = torch.empty(shape, dtype=d["k"].dtype, device=gpu)
    v_out = torch.empty_like(k_out)
    scores = torch.empty((w.n_kv_heads, p.total_tokens), dtype=torch.float32, device=gpu)
    ws = C.workspace(p, d["srh_mask"], B, gpu)
    outs = [idx, k_out, v_out, scores]

    def call():
        C.compresskv_compress_layer(p, d["q_win"], d["k"], d["v"], d["srh_mask"], B, idx, k_out,
                                    v_out, scores, ws)

    call()
    torch.cuda.synchronize()
    ref = [t.clone() for t in outs]
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call()
    torch.cuda.synchronize()
    _replays_match(g, outs, ref, gpu)
