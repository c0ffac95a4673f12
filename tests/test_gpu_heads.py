"""GPU parity of the per-group (head-level) budgets against the oracle's
compress_layer_heads: ragged per-group outputs, under the acceptance rules of
tests/parity_helpers.py applied group by group."""
import sys

import numpy as np
import pytest
import torch

import oracle as O
from paper_2606_24467_amd import compresskv as C
from paper_2606_24467_amd import workloads as wl
from tests import parity_helpers as H

pytestmark = pytest.mark.gpu


@pytest.fixture(autouse=True)
def _two_pass(monkeypatch):
    monkeypatch.delenv("CKV_PATH", raising=False)


def _say(*a):
    print(*a, file=sys.stderr, flush=True)


def _check(x, budgets, got, ora):
    idx, k_out, v_out, scores = got
    cu, W = x.cu_seqlens, x.workload.window
    H.check_scores(scores, ora, cu, W)
    off = np.concatenate([[0], np.cumsum(budgets)])
    Hkv = len(budgets)
    kb = x.bits("k") if x.dtype == wl.BF16 else x.k.view(np.uint32)
    vb = x.bits("v") if x.dtype == wl.BF16 else x.v.view(np.uint32)
    swaps = 0
    for g, B in enumerate(budgets):
        # one group at a time, in the fixed-budget layout the helpers expect
        sl = slice(int(off[g]), int(off[g + 1]))
        gi = np.full((idx.shape[0], Hkv, B), -1, dtype=idx.dtype)
        gi[:, g] = idx[:, sl]
        oi = O.LayerResult(idx=np.full((idx.shape[0], Hkv, B), -1), k_out=None, v_out=None,
                           scores=ora.scores)
        oi.idx[:, g] = ora.idx[:, sl]
        swaps += H.check_indices(gi, oi, cu, W, B, groups=[g])
        ko = np.zeros((idx.shape[0], Hkv, B) + k_out.shape[2:], dtype=k_out.dtype)
        vo = np.zeros_like(ko)
        ko[:, g] = k_out[:, sl]
        vo[:, g] = v_out[:, sl]
        H.check_gather(ko, vo, gi, kb, vb, cu, groups=[g])
    return swaps


@pytest.mark.parametrize("name,budgets_fn", [
    ("ragged budgets", lambda W, L: [W, 3 * W, 257, 2000, 64, W + 1, 700, 90]),
    ("equal budgets", lambda W, L: [300] * 8),
])
def test_compress_layer_heads_matches_oracle(gpu, name, budgets_fn):
    w = wl.get("ragged8", batch=3, ragged=(600, 2200), srh_per_group=(1, 2), n_needle=4)
    x = wl.make_layer(w, 0, seed=41, budget=64)
    budgets = budgets_fn(w.window, None)
    _say(f"case heads {name} L={np.diff(x.cu_seqlens).tolist()} budgets={budgets}")
    q, k, v, cu = H.device_tensors(x, gpu)
    p = C.Problem(q, k, v, cu, cu_seqlens_host=x.cu_seqlens, pool_kernel=w.pool_kernel,
                  pool_type=w.pool_type)
    idx, k_out, v_out, scores = C.compress_layer_heads(p, q, k, v, x.srh_mask, budgets,
                                                       want_scores=True)
    torch.cuda.synchronize()
    kb = x.bits("k") if x.dtype == wl.BF16 else x.k.view(np.uint32)
    vb = x.bits("v") if x.dtype == wl.BF16 else x.v.view(np.uint32)
    ora = O.compress_layer_heads(x.q_win, kb, vb, x.cu_seqlens, x.srh_mask, budgets,
                                 w.pool_kernel, w.pool_type, k_values=x.k)
    got = (idx.cpu().numpy(), H.raw_bits(k_out), H.raw_bits(v_out), scores.cpu().numpy())
    swaps = _check(x, budgets, got, ora)
    _say(f"  ok, boundary swaps {swaps}")
    if name == "equal budgets":
        ref = C.compress_layer(p, q, k, v, x.srh_mask, 300, want_scores=True)
        torch.cuda.synchronize()
        assert torch.equal(idx, ref[0].reshape(idx.shape))
        assert torch.equal(k_out, ref[1].reshape(k_out.shape))


def test_select_and_gather_heads_entry_points(gpu):
    """select_heads / gather_heads one after the other give the same bits as
    compress_layer_heads."""
    w = wl.get("llama1", seq_len=4000 + 7, n_needle=4)
    x = wl.make_layer(w, 0, seed=42)
    budgets = [40 + 37 * g for g in range(w.n_kv_heads)]
    q, k, v, cu = H.device_tensors(x, gpu)
    p = C.Problem(q, k, v, cu, cu_seqlens_host=x.cu_seqlens)
    ref = C.compress_layer_heads(p, q, k, v, x.srh_mask, budgets, want_scores=True)
    scores = C.score(p, q, k, x.srh_mask)
    total = sum(budgets)
    idx = torch.empty((1, total), dtype=torch.int32, device=gpu)
    C.compresskv_select_heads(p, scores, budgets, idx)
    k_out = torch.empty((1, total, w.head_dim), dtype=k.dtype, device=gpu)
    v_out = torch.empty_like(k_out)
    C.compresskv_gather_heads(p, k, v, idx, budgets, k_out, v_out)
    torch.cuda.synchronize()
    for got, want in zip((idx, k_out, v_out, scores), ref):
        assert torch.equal(got, want)
