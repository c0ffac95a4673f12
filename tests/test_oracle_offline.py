"""Pins of the offline oracle (oracle/offline_oracle.py): the SRH score of
equation 1 and the per-layer top-k, the eviction error of equations 2-4 and
the layer budget allocation.  Every pin is independent of the oracle's code:
hand-worked fractions (tests/golden), closed forms, a batched torch
computation, and invariants."""
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import torch

from oracle import offline_oracle as OO

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    rows = {}
    for line in open(os.path.join(GOLDEN, name)):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        key, *vals = line.split()
        rows.setdefault(key, []).append(vals)
    return rows


# ---------------------------------------------------------------- equation 1
def test_srh_score_hand_worked_example():
    g = _golden("srh_worked.txt")
    ctx = np.array([int(x) for x in g["ctx"][0]])
    a0, n = (int(x) for x in g["span"][0])
    gen = np.array([int(x) for x in g["gen"][0]])
    attn = np.zeros((1, 3, 2, 5))
    for row in g["attn"]:
        t, h = int(row[0]), int(row[1])
        attn[0, t, h] = [float(Fraction(x)) for x in row[2:]]
    got = OO.srh_scores(attn, gen[None], ctx[None], np.array([[a0, n]]))
    want = [float(Fraction(x)) for x in g["scores"][0]]
    np.testing.assert_allclose(got, want, rtol=1e-15)
    mask = OO.select_srh(got, 1, 1)
    assert mask[0].tolist() == [1 if h == int(g["top1"][0][0]) else 0 for h in range(2)]


def _random_calibration(seed, S=3, N=7, H=12, L=40):
    rng = np.random.default_rng(seed)
    logits = rng.standard_normal((S, N, H, L)) * 2
    attn = np.exp(logits)
    attn /= attn.sum(-1, keepdims=True)
    ctx = rng.integers(0, 30, size=(S, L))
    spans = np.stack([rng.integers(0, L - 6, size=S), rng.integers(1, 6, size=S)], 1)
    gen = rng.integers(0, 30, size=(S, N))
    for s in range(S):   # make some steps hit the answer
        gen[s, ::2] = ctx[s, spans[s, 0]]
    return attn, gen, ctx, spans


def test_srh_score_equals_masked_einsum():
    """sum_s,t,j hit[s,t] * in_span[s,j] * a[s,t,h,j] with the masks built by
    np.isin and index ranges."""
    attn, gen, ctx, spans = _random_calibration(1)
    S, N, H, L = attn.shape
    span_mask = np.zeros((S, L))
    hits = np.zeros((S, N))
    for s in range(S):
        span_mask[s, spans[s, 0]:spans[s, 0] + spans[s, 1]] = 1
        hits[s] = np.isin(gen[s], ctx[s, spans[s, 0]:spans[s, 0] + spans[s, 1]])
    want = np.einsum("sthj,sj,st->h", attn, span_mask, hits)
    np.testing.assert_allclose(OO.srh_scores(attn, gen, ctx, spans), want, rtol=1e-12)


def test_srh_score_closed_forms():
    S, N, H, L = 2, 5, 3, 20
    ctx = np.tile(np.arange(L), (S, 1))
    spans = np.array([[4, 3], [10, 5]])
    gen = np.array([[4, 0, 5, 6, 19], [10, 11, 0, 0, 14]])   # hits 3 and 3
    uniform = np.full((S, N, H, L), 1.0 / L)
    # uniform attention: hits * span length / L
    np.testing.assert_allclose(OO.srh_scores(uniform, gen, ctx, spans),
                               [(3 * 3 + 3 * 5) / L] * H, rtol=1e-14)
    # one-hot attention on a span position at every step: the number of hits
    onehot = np.zeros((S, N, H, L))
    onehot[0, :, :, 5] = 1
    onehot[1, :, :, 12] = 1
    np.testing.assert_allclose(OO.srh_scores(onehot, gen, ctx, spans), [6.0] * H, rtol=0)
    # no step generates an answer token: zero
    assert np.all(OO.srh_scores(uniform, np.full((S, N), 99), ctx, spans) == 0)


def test_srh_score_is_linear_and_ignores_other_positions():
    attn, gen, ctx, spans = _random_calibration(2)
    base = OO.srh_scores(attn, gen, ctx, spans)
    np.testing.assert_allclose(OO.srh_scores(3 * attn, gen, ctx, spans), 3 * base, rtol=1e-13)
    other = attn.copy()
    for s in range(attn.shape[0]):
        a0, n = spans[s]
        other[s, :, :, :a0] *= 7
        other[s, :, :, a0 + n:] = 0
    np.testing.assert_allclose(OO.srh_scores(other, gen, ctx, spans), base, rtol=1e-13)


def test_select_srh_ranks_each_layer_with_lowest_index_ties():
    scores = np.array([0.5, 0.9, 0.9, 0.1,   0.2, 0.2, 0.2, 0.3])
    m = OO.select_srh(scores, 2, 2)
    assert m.tolist() == [[0, 1, 1, 0], [1, 0, 0, 1]]
    assert OO.select_srh(scores, 2, 4).sum() == 8
    rng = np.random.default_rng(3)
    sc = rng.standard_normal(6 * 32)
    m = OO.select_srh(sc, 6, 4)
    for l in range(6):
        want = np.argsort(-sc[l * 32:(l + 1) * 32], kind="stable")[:4]
        assert sorted(np.flatnonzero(m[l]).tolist()) == sorted(want.tolist())


# ---------------------------------------------------------- equations 2 - 4
def _decode_case(seed, batch=2, T=3, Hq=8, Hkv=2, D=16, lens=(60, 45), B=12, d_model=24):
    rng = np.random.default_rng(seed)
    cu = np.concatenate([[0], np.cumsum(lens)])
    k = rng.standard_normal((cu[-1], Hkv, D))
    v = rng.standard_normal((cu[-1], Hkv, D))
    q = rng.standard_normal((batch, T, Hq, D))
    idx = np.full((batch, Hkv, B), -1)
    for b in range(batch):
        L = lens[b]
        for g in range(Hkv):
            keep = np.sort(rng.choice(L, size=min(B, L) - 2, replace=False))
            idx[b, g, :len(keep)] = keep
    w_o = rng.standard_normal((d_model, Hq * D))
    return q, k, v, cu, idx, w_o


def _torch_error(q, k, v, cu, idx, w_o, eps):
    """The same error with batched torch attention over masked logits."""
    batch, T, Hq, D = q.shape
    Hkv = k.shape[1]
    G = Hq // Hkv
    W = torch.from_numpy(w_o)
    total = 0.0
    for b in range(batch):
        s0, s1 = int(cu[b]), int(cu[b + 1])
        L = s1 - s0
        kt = torch.from_numpy(k[s0:s1]).permute(1, 0, 2).repeat_interleave(G, 0)   # [Hq, L, D]
        vt = torch.from_numpy(v[s0:s1]).permute(1, 0, 2).repeat_interleave(G, 0)
        qt = torch.from_numpy(q[b]).permute(1, 0, 2)                                 # [Hq, T, D]
        z = torch.matmul(qt, kt.transpose(1, 2).contiguous()) / math.sqrt(D)        # [Hq, T, L]
        keep = torch.zeros((Hq, 1, L), dtype=torch.bool)
        for h in range(Hq):
            sel = idx[b, h // G]
            keep[h, 0, torch.from_numpy(sel[sel >= 0])] = True
        full = torch.matmul(torch.softmax(z, -1), vt)                                 # [Hq, T, D]
        comp = torch.matmul(torch.softmax(z.masked_fill(~keep, float("-inf")), -1), vt)
        for t in range(T):
            of = W @ full[:, t].reshape(-1)
            od = W @ (full[:, t] - comp[:, t]).reshape(-1)
            total += float(torch.linalg.norm(od) / (torch.linalg.norm(of) + eps))
    return total


def test_layer_error_matches_batched_torch():
    q, k, v, cu, idx, w_o = _decode_case(4)
    got = OO.layer_error(q, k, v, cu, idx, w_o)
    np.testing.assert_allclose(got, _torch_error(q, k, v, cu, idx, w_o, 1e-6), rtol=1e-10)


def test_layer_error_closed_forms():
    q, k, v, cu, idx, w_o = _decode_case(5, lens=(30, 20), B=40)
    # every position kept: the compressed output is the full one
    full_idx = np.full(idx.shape, -1)
    for b in range(2):
        L = int(cu[b + 1] - cu[b])
        full_idx[b, :, :L] = np.arange(L)
    assert OO.layer_error(q, k, v, cu, full_idx, w_o) == 0.0
    # one kept key per group: that head's compressed output is the kept V row;
    # with W_O = I the error is ||A_full - V_kept|| / (||A_full|| + eps)
    q1, k1, v1 = q[:1, :1, :2], k[:30, :1], v[:30, :1]
    one = np.full((1, 1, 4), -1)
    one[0, 0, 0] = 7
    D = q1.shape[-1]
    e = OO.layer_error(q1, k1, v1, np.array([0, 30]), one, np.eye(2 * D), eps=0.0)
    z = (k1[:, 0] @ q1[0, 0].T) / math.sqrt(D)          # [30, 2]
    w = np.exp(z - z.max(0))
    w /= w.sum(0)
    a = (w.T @ v1[:, 0])                                 # [2, D]
    want = np.linalg.norm(a - v1[7, 0][None]) / np.linalg.norm(a)
    np.testing.assert_allclose(e, want, rtol=1e-12)


def test_layer_error_invariants():
    q, k, v, cu, idx, w_o = _decode_case(6)
    e = OO.layer_error(q, k, v, cu, idx, w_o, eps=0.0)
    # a scaled projection leaves the relative error unchanged
    np.testing.assert_allclose(OO.layer_error(q, k, v, cu, idx, 5 * w_o, eps=0.0), e, rtol=1e-12)
    # an orthogonal projection keeps every norm: same error as no projection
    Qm, _ = np.linalg.qr(np.random.default_rng(7).standard_normal((w_o.shape[1],) * 2))
    np.testing.assert_allclose(OO.layer_error(q, k, v, cu, idx, Qm, eps=0.0),
                               OO.layer_error(q, k, v, cu, idx, np.eye(w_o.shape[1]), eps=0.0),
                               rtol=1e-10)
    # sequences and steps add up
    parts = sum(OO.layer_error(q[b:b + 1, t:t + 1], k[cu[b]:cu[b + 1]], v[cu[b]:cu[b + 1]],
                               np.array([0, cu[b + 1] - cu[b]]), idx[b:b + 1], w_o, eps=0.0)
                for b in range(2) for t in range(q.shape[1]))
    np.testing.assert_allclose(parts, e, rtol=1e-12)


# ----------------------------------------------------------- layer budgets
def test_budget_hand_worked_example():
    g = _golden("budget_worked.txt")
    e = np.array([float(x) for x in g["errors"][0]])
    # equation 4's normalisation: each error over the sum of all of them
    want = [Fraction(x) for x in g["normalised"][0]]
    got_n = OO.normalize_errors(e)
    assert np.allclose(got_n, [float(x) for x in want], rtol=0, atol=1e-15)
    got = OO.allocate_budgets(OO.normalize_errors(e), int(g["total"][0][0]),
                              int(g["min"][0][0]), int(g["max"][0][0]))
    assert got.tolist() == [int(x) for x in g["budgets"][0]]


def test_budget_closed_forms():
    # exact proportional split when nothing is capped and shares are integral
    assert OO.allocate_budgets(np.array([0.1, 0.2, 0.3, 0.4]), 4 * 32 + 100, 32, 1000).tolist() \
        == [42, 52, 62, 72]
    # rounding: shares 10/7, 20/7, 40/7 floor to 1, 2, 5; the two units left go
    # to the largest fractional parts (6/7 and 5/7), not to the first layers
    assert OO.allocate_budgets(np.array([1, 2, 4]) / 7, 3 * 32 + 10, 32, 1000).tolist() == \
        [33, 35, 38]
    # equal errors: an even split, the remainder to the lowest layers
    assert OO.allocate_budgets(np.full(4, 0.25), 4 * 32 + 10, 32, 1000).tolist() == \
        [35, 35, 34, 34]
    # total at the bounds
    assert OO.allocate_budgets(np.array([0.7, 0.2, 0.1]), 3 * 32, 32, 96).tolist() == [32] * 3
    assert OO.allocate_budgets(np.array([0.7, 0.2, 0.1]), 3 * 96, 32, 96).tolist() == [96] * 3


@pytest.mark.parametrize("seed", range(4))
def test_normalised_errors_are_shares(seed):
    """e~ is a distribution over the layers: non-negative, summing to one, in
    the same ratios as e (exactly, for integer errors, via fractions)."""
    rng = np.random.default_rng(100 + seed)
    e = rng.integers(1, 1000, size=int(rng.integers(2, 40))).astype(np.float64)
    got = OO.normalize_errors(e)
    assert abs(got.sum() - 1.0) < 1e-12 and np.all(got >= 0)
    tot = sum(Fraction(int(x)) for x in e)
    for x, y in zip(e, got):
        assert abs(Fraction(int(x)) / tot - Fraction(float(y))) < Fraction(1, 10**14)
    # scaling every error leaves the shares unchanged
    np.testing.assert_allclose(OO.normalize_errors(7.5 * e), got, rtol=1e-14)


@pytest.mark.parametrize("seed", range(6))
def test_budget_invariants(seed):
    """The paper's setting: m = 32, M = 3 x the per-layer average."""
    rng = np.random.default_rng(seed)
    n, per = 32, int(rng.integers(64, 2049))
    e = rng.gamma(0.5, size=n)
    b = OO.allocate_budgets(OO.normalize_errors(e), n * per, 32, 3 * per)
    assert b.sum() == n * per and b.min() >= 32 and b.max() <= 3 * per
    order = np.argsort(e)
    assert np.all(np.diff(b[order]) >= -1)       # monotone up to one rounding unit
    free = b < 3 * per
    # uncapped layers: within one unit of the proportional share of what is left
    rest = n * per - b[~free].sum() - 32 * free.sum()
    share = rest * e[free] / e[free].sum()
    assert np.all(np.abs(b[free] - 32 - share) < 1.0)
