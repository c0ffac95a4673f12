"""The selection split over slices of 32768 prefix positions (per-group index
sets of sequences longer than one slice): its kept lists are exactly the
oracle's selection on the same fp32 scores (section 3.3: the best prefix
tokens by score, ties to the lowest position, plus the window), across
ragged lengths, budgets, ties that straddle a slice boundary, buckets
holding every position, multi-layer calls and per-group budgets."""
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


def _check_exact(scores, idx_rows, cu, W, budgets):
    """idx_rows(b, g) -> the kept list; budgets[g] the group's budget."""
    for b in range(len(cu) - 1):
        s0, s1 = int(cu[b]), int(cu[b + 1])
        L = s1 - s0
        for g in range(scores.shape[0]):
            want = O.select_tokens(scores[g, s0:s1 - W].astype(np.float64), L, W, budgets[g])
            got = idx_rows(b, g)
            n = len(want)
            assert np.array_equal(got[:n], want), (b, g, L, budgets[g])
            assert np.all(got[n:] == -1), (b, g)


def _layer(lengths, seed, **kw):
    w = wl.get("llama1", batch=len(lengths), **kw)
    return wl.make_layer(w, 0, seed=seed, lengths=np.asarray(lengths))


def test_split_select_ragged_lengths_and_budgets(gpu):
    # prefixes of 3 slices, under one slice, exactly one slice, 2 slices
    x = _layer([70000, 5000, 32800, 40000], seed=31)
    W = x.workload.window
    q, k, v, cu = H.device_tensors(x, gpu)
    p = C.Problem(q, k, v, cu, cu_seqlens_host=x.cu_seqlens, scoring=C.SCORE_TWO_PASS)
    for budget in (W, W + 1, 1024, 33000, 50000):
        _say(f"case ragged split select, budget {budget}")
        idx, _, _, scores = C.compress_layer(p, q, k, v, x.srh_mask, budget, want_scores=True)
        torch.cuda.synchronize()
        idx, scores = idx.cpu().numpy(), scores.cpu().numpy()
        _check_exact(scores, lambda b, g: idx[b, g], x.cu_seqlens, W, [budget] * 8)
    ora = H.run_oracle(x, 1024)
    idx, ko, vo, scores = C.compress_layer(p, q, k, v, x.srh_mask, 1024, want_scores=True)
    torch.cuda.synchronize()
    H.check_scores(scores.cpu().numpy(), ora, x.cu_seqlens, W)
    H.check_indices(idx.cpu().numpy(), ora, x.cu_seqlens, W, 1024)
    H.check_gather(H.raw_bits(ko), H.raw_bits(vo), idx.cpu().numpy(), x.bits("k"), x.bits("v"),
                   x.cu_seqlens)


def _plant_block(x, g, start, n, alpha):
    """n equal keys at [start, start + n) of group g of sequence 0, along the
    group's mean SRH query direction: after max pooling a plateau of equal
    scores over [start - r, start + n + r)."""
    w = x.workload
    G = w.n_q_heads // w.n_kv_heads
    heads = [h for h in range(g * G, (g + 1) * G) if x.srh_mask[h]]
    d = x.q_win[0][:, heads, :].astype(np.float64).mean(axis=(0, 1))
    d = d / np.linalg.norm(d)
    vec = (alpha * np.sqrt(w.head_dim) * d).astype(np.float32)
    vec = wl.bf16_bits_to_f32(wl.f32_to_bf16_bits(vec))
    x.k[start:start + n, g, :] = vec


def test_split_select_ties_straddling_a_slice_boundary(gpu):
    """Group 0: one plateau over positions 32757-32778 (slice boundary at
    32768) and a budget that keeps 15 of its ties, 11 before the boundary
    and 4 after.  Group 1: a higher plateau inside the second slice and the
    same straddling plateau, with a budget that keeps all of the first and
    the lowest 5 ties of the second, so the second slice's kept list starts
    after the first slice's ties."""
    x = _layer([70000], seed=32, n_needle=0, n_sink=0)
    W, r = x.workload.window, x.workload.pool_kernel // 2
    _plant_block(x, 0, 32760, 16, 4.0)
    _plant_block(x, 1, 32760, 16, 4.0)
    _plant_block(x, 1, 40000, 16, 6.0)
    q, k, v, cu = H.device_tensors(x, gpu)
    p = C.Problem(q, k, v, cu, cu_seqlens_host=x.cu_seqlens, scoring=C.SCORE_TWO_PASS)
    budgets = [W + 15, W + 22 + 5] + [W + 100] * 6
    idx, _, _, scores = C.compress_layer_heads(p, q, k, v, x.srh_mask, budgets, want_scores=True)
    torch.cuda.synchronize()
    idx, scores = idx.cpu().numpy(), scores.cpu().numpy()
    lo, hi = 32760 - r, 32760 + 16 + r
    for g in (0, 1):
        plateau = scores[g, lo:hi]
        assert np.all(plateau == plateau[0]), f"group {g}: the planted plateau is not flat"
        assert plateau[0] > scores[g, lo - 1] and plateau[0] > scores[g, hi]
    off = np.concatenate([[0], np.cumsum(budgets)])
    _check_exact(scores, lambda b, g: idx[b, off[g]:off[g + 1]], x.cu_seqlens, W, budgets)
    assert idx[0, :15].tolist() == list(range(lo, lo + 15))
    assert idx[0, off[1]:off[1] + 27].tolist() == (list(range(lo, lo + 5)) +
                                                    list(range(40000 - r, 40016 + r)))
    # the same kept lists from the one-workgroup selection of compresskv_select_heads
    idx1 = torch.empty((1, int(off[-1])), dtype=torch.int32, device=gpu)
    C.compresskv_select_heads(p, torch.from_numpy(scores).to(gpu), budgets, idx1)
    torch.cuda.synchronize()
    assert np.array_equal(idx1.cpu().numpy(), idx)


def test_split_select_full_bucket(gpu):
    """Constant keys: every prefix score is equal, each slice's bucket holds
    all of its 32768 positions (more candidates than the resolve kernel keeps
    in LDS, and every position in the slice's ordered list), and the lowest
    positions are kept."""
    x = _layer([70000, 40000], seed=33, n_needle=0, n_sink=0)
    x.k[:] = 0.0
    W = x.workload.window
    q, k, v, cu = H.device_tensors(x, gpu)
    p = C.Problem(q, k, v, cu, cu_seqlens_host=x.cu_seqlens, scoring=C.SCORE_TWO_PASS)
    for budget in (W + 1000, W + 36000):
        idx, _, _, scores = C.compress_layer(p, q, k, v, x.srh_mask, budget, want_scores=True)
        torch.cuda.synchronize()
        idx, scores = idx.cpu().numpy(), scores.cpu().numpy()
        _check_exact(scores, lambda b, g: idx[b, g], x.cu_seqlens, W, [budget] * 8)
        assert idx[0, 0, :budget - W].tolist() == list(range(budget - W))


def test_split_select_multi_layer_ragged_batch(gpu):
    """A multi-layer call over a ragged batch whose sequences span 3, 1 and 2
    slices, with a different budget per layer: every layer's kept lists are
    exactly the oracle's selection on its fp32 scores and equal the
    per-layer call's bit for bit."""
    w = wl.get("llama1", batch=3, n_layers=3, n_needle=4)
    lengths = np.asarray([70000, 5000, 40000])
    xs = [wl.make_layer(w, l, seed=34, lengths=lengths) for l in range(w.n_layers)]
    W = w.window
    budgets = [1024, W + 3, 36000]
    dts = [H.device_tensors(x, gpu) for x in xs]
    q, k, v = [d[0] for d in dts], [d[1] for d in dts], [d[2] for d in dts]
    cu = dts[0][3]
    masks = np.stack([x.srh_mask for x in xs])
    p = C.Problem(q[0], k[0], v[0], cu, cu_seqlens_host=xs[0].cu_seqlens,
                  scoring=C.SCORE_TWO_PASS)
    _say(f"case multi-layer split select, lengths {lengths.tolist()}, budgets {budgets}")
    idxs, kos, vos, scores = C.compress_layers(p, q, k, v, masks, budgets, want_scores=True)
    torch.cuda.synchronize()
    for l in range(w.n_layers):
        il, sl = idxs[l].cpu().numpy(), scores[l].cpu().numpy()
        _check_exact(sl, lambda b, g: il[b, g], xs[0].cu_seqlens, W, [budgets[l]] * 8)
        pl = C.Problem(q[l], k[l], v[l], cu, cu_seqlens_host=xs[0].cu_seqlens,
                       scoring=C.SCORE_TWO_PASS)
        one = C.compress_layer(pl, q[l], k[l], v[l], masks[l], budgets[l], want_scores=True)
        torch.cuda.synchronize()
        for got, want in zip((idxs[l], kos[l], vos[l], scores[l]), one):
            assert torch.equal(got, want), f"layer {l} differs from the per-layer call"


def test_split_select_heads_ragged_batch(gpu):
    """Per-group budgets (compress_layer_heads) over a ragged batch longer
    than one slice: budgets from the window alone to more than a slice and
    more than the shorter sequence, kept lists exactly the oracle's selection
    on the fp32 scores, kept rows equal to the keys and values at those
    positions."""
    x = _layer([70000, 40000], seed=35, n_needle=4)
    W = x.workload.window
    q, k, v, cu = H.device_tensors(x, gpu)
    p = C.Problem(q, k, v, cu, cu_seqlens_host=x.cu_seqlens, scoring=C.SCORE_TWO_PASS)
    budgets = [W, 3000, 257, 36000, 64, W + 1, 45000, 12000]
    _say(f"case heads split select, budgets {budgets}")
    idx, k_out, v_out, scores = C.compress_layer_heads(p, q, k, v, x.srh_mask, budgets,
                                                       want_scores=True)
    torch.cuda.synchronize()
    idx, scores = idx.cpu().numpy(), scores.cpu().numpy()
    off = np.concatenate([[0], np.cumsum(budgets)])
    _check_exact(scores, lambda b, g: idx[b, off[g]:off[g + 1]], x.cu_seqlens, W, budgets)
    kb, vb = x.bits("k"), x.bits("v")
    ko, vo = H.raw_bits(k_out), H.raw_bits(v_out)
    for b in range(2):
        s0 = int(x.cu_seqlens[b])
        for g in range(8):
            rows = idx[b, off[g]:off[g + 1]]
            kept = rows >= 0
            assert np.array_equal(ko[b, off[g]:off[g + 1]][kept], kb[s0 + rows[kept], g])
            assert np.array_equal(vo[b, off[g]:off[g + 1]][kept], vb[s0 + rows[kept], g])
            assert not ko[b, off[g]:off[g + 1]][~kept].any()
