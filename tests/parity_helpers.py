"""Shared helpers of the parity tests: move generator inputs to the GPU, run
the oracle on the same values, and apply the acceptance rules.

Acceptance (per sequence b and KV group g):
  * scores: |gpu - oracle| <= 2e-3 * max(|oracle|, 1e-6 * max_j oracle_j) on
    prefix positions, +inf on window positions;
  * indices: the same count; any position kept by only one side must have an
    oracle score within 1e-5 (relative) of the oracle's kept threshold tau,
    the (budget - W)-th largest prefix score;
  * gathered K/V: bit-identical to K[cu_b + idx_gpu] / V[...] for every kept
    row (so bit-identical to the oracle wherever indices agree), zeros on -1.
"""
from __future__ import annotations

import numpy as np
import torch

import oracle as O
from paper_2606_24467_amd import workloads as wl

SCORE_RTOL = 2e-3
BOUNDARY_RTOL = 1e-5

# Scoring path of the problems the GPU tests build (ckv_problem.scoring); the
# parametrised fixtures of the parity test files set it per case.
SCORING = 0


def problem(q, k, v, cu, *, masks=None, **kw):
    """A C.Problem on the scoring path SCORING.  With the single pass forced,
    a problem (or a layer mask) it does not apply to skips the case."""
    import pytest
    from paper_2606_24467_amd import compresskv as C
    kw.setdefault("scoring", SCORING)
    p = C.Problem(q, k, v, cu, **kw)
    if masks is not None and p.c.scoring == C.SCORE_ONE_PASS:
        for m in np.atleast_2d(np.asarray(masks)):
            try:
                C.compresskv_scoring_path(p, m)
            except C.CompressKVError as e:
                if e.status != C.UNSUPPORTED:
                    raise
                pytest.skip(f"the single pass does not apply: {e}")
    return p


def device_tensors(x: wl.LayerInputs, dev):
    """q_win, k, v, cu_seqlens as device tensors holding exactly x's values."""
    def t(name):
        a = x.bits(name)
        if x.dtype == wl.BF16:
            return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).to(dev).view(
                torch.bfloat16)
        return torch.from_numpy(np.ascontiguousarray(a)).to(dev)
    cu = torch.from_numpy(x.cu_seqlens.astype(np.int32)).to(dev)
    return t("q_win"), t("k"), t("v"), cu


def run_oracle(x: wl.LayerInputs, budget=None, pool_kernel=None, pool_type=None,
               reduce_order=O.POOL_THEN_MEAN, scale=None,
               index_mode=O.PER_GROUP) -> O.LayerResult:
    w = x.workload
    kb = x.bits("k") if x.dtype == wl.BF16 else x.k.view(np.uint32)
    vb = x.bits("v") if x.dtype == wl.BF16 else x.v.view(np.uint32)
    return O.compress_layer(x.q_win, kb, vb, x.cu_seqlens, x.srh_mask,
                            x.budget if budget is None else budget,
                            w.pool_kernel if pool_kernel is None else pool_kernel,
                            w.pool_type if pool_type is None else pool_type,
                            reduce_order, scale=scale, k_values=x.k, index_mode=index_mode)


def raw_bits(t: torch.Tensor) -> np.ndarray:
    """Device tensor -> host array of its raw bits (uint16 for bf16, uint32 for fp32)."""
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).cpu().numpy().view(np.uint16)
    return t.contiguous().cpu().numpy().view(np.uint32)


def check_scores(gpu_scores: np.ndarray, ora: O.LayerResult, cu, W, groups=None):
    Hkv = gpu_scores.shape[0]
    for b in range(len(cu) - 1):
        s0, s1 = int(cu[b]), int(cu[b + 1])
        P = s1 - s0 - W
        for g in (range(Hkv) if groups is None else groups):
            o = ora.scores[g, s0:s0 + P]
            gsc = gpu_scores[g, s0:s0 + P].astype(np.float64)
            assert np.all(np.isinf(gpu_scores[g, s0 + P:s1])), f"window not +inf (b={b}, g={g})"
            if P == 0:
                continue
            floor = 1e-6 * float(np.max(o))
            tol = SCORE_RTOL * np.maximum(np.abs(o), floor)
            err = np.abs(gsc - o)
            bad = np.nonzero(err > tol)[0]
            assert bad.size == 0, (f"scores differ (b={b}, g={g}) at {bad[:8]}: gpu "
                                   f"{gsc[bad[:8]]} oracle {o[bad[:8]]}")


def check_indices(gpu_idx: np.ndarray, ora: O.LayerResult, cu, W, budget, groups=None):
    """Returns the number of boundary swaps that were accepted."""
    swaps = 0
    Hkv = gpu_idx.shape[1]
    for b in range(len(cu) - 1):
        s0, s1 = int(cu[b]), int(cu[b + 1])
        L = s1 - s0
        P = L - W
        n = min(budget, L)
        for g in (range(Hkv) if groups is None else groups):
            gi = gpu_idx[b, g]
            oi = ora.idx[b, g]
            assert np.all(gi[n:] == -1), f"padding not -1 (b={b}, g={g})"
            sel_g = gi[:n]
            assert np.all(np.diff(sel_g) > 0), f"indices not ascending/unique (b={b}, g={g})"
            assert np.all((sel_g >= 0) & (sel_g < L))
            if np.array_equal(sel_g, oi[:n]):
                continue
            assert L > budget
            o = ora.scores[g, s0:s0 + P]
            k = budget - W
            tau = np.sort(o)[::-1][k - 1]
            diff = np.setxor1d(sel_g, oi[:n])
            assert np.all(diff < P), f"window positions differ (b={b}, g={g})"
            rel = np.abs(o[diff] - tau) / tau
            assert np.all(rel <= BOUNDARY_RTOL), (
                f"index mismatch beyond the boundary tolerance (b={b}, g={g}): positions "
                f"{diff[:8]} oracle scores {o[diff[:8]]} tau {tau}")
            swaps += diff.size // 2
    return swaps


def check_gather(k_out: np.ndarray, v_out: np.ndarray, gpu_idx: np.ndarray, kbits, vbits, cu,
                 groups=None):
    Hkv = gpu_idx.shape[1]
    for b in range(len(cu) - 1):
        s0 = int(cu[b])
        for g in (range(Hkv) if groups is None else groups):
            sel = gpu_idx[b, g]
            keep = sel >= 0
            np.testing.assert_array_equal(k_out[b, g][keep], kbits[s0 + sel[keep], g])
            np.testing.assert_array_equal(v_out[b, g][keep], vbits[s0 + sel[keep], g])
            assert np.all(k_out[b, g][~keep] == 0) and np.all(v_out[b, g][~keep] == 0)
