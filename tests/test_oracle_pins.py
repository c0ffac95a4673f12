"""Pins of the fp64 oracle against things other than itself.

Each test ties one step of the oracle (section 3.3 token selection with the
SnapKV window setting of section 4) to a hand-worked fraction example, an
exact rational brute force, a scalar brute-force attention, a library routine,
a closed form, an invariant or a metamorphic relation.
"""
import math
import os
import random
from fractions import Fraction

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ------------------------------------------------------------------ helpers
def _layer(q_heads, keys, W, budget, pool_kernel, pool_type, reduce_order=O.POOL_THEN_MEAN,
           scale=None):
    """Run oracle.compress_layer on one sequence, one group, given SRH queries."""
    n = len(q_heads)
    L, D = keys.shape
    q = np.stack(q_heads, axis=1)[None]            # [1, W, n, D]
    k = keys[:, None, :].copy()
    v = np.arange(L * D, dtype=np.float64).reshape(L, 1, D)
    mask = np.ones(n, dtype=np.uint8)
    return O.compress_layer(q, k, v, np.array([0, L]), mask, budget, pool_kernel,
                            pool_type, reduce_order, scale=scale)


def _parse_golden(path):
    spec = {"query_exp": []}
    for line in open(path):
        line = line.strip()
        if not line or line.startswith("#"):
            continue
        key, *vals = line.split()
        if key == "query_exp":
            spec["query_exp"].append([int(x) for x in vals])
        elif key in ("colsum", "scores"):
            spec[key] = [Fraction(x) for x in vals]
        elif key == "pool":
            spec["pool"] = (O.POOL_MAX if vals[0] == "max" else O.POOL_AVG, int(vals[1]))
        elif key in ("keys_exp", "selected"):
            spec[key] = [int(x) for x in vals]
        else:
            spec[key] = int(vals[0])
    return spec


# --------------------------------------------------- hand-worked fractions
@pytest.mark.parametrize("name", ["worked_max3.txt", "worked_avg3.txt", "worked_two_heads.txt"])
def test_hand_worked_examples(name):
    spec = _parse_golden(os.path.join(GOLDEN, name))
    W = spec["window"]
    keys = np.log(np.array(spec["keys_exp"], dtype=np.float64))[:, None]
    q_heads = [np.array(q, dtype=np.float64)[:, None] for q in spec["query_exp"]]
    kind, kernel = spec["pool"]
    res = _layer(q_heads, keys, W, spec["budget"], kernel, kind, scale=1.0)
    P = keys.shape[0] - W
    if "colsum" in spec:
        a = O.row_softmax(O.window_logits(q_heads[0], keys, 1.0))
        np.testing.assert_allclose(O.window_column_sums(a, P),
                                   [float(x) for x in spec["colsum"]], rtol=1e-13, atol=0)
    np.testing.assert_allclose(res.scores[0, :P], [float(x) for x in spec["scores"]],
                               rtol=1e-13, atol=0)
    assert np.all(np.isinf(res.scores[0, P:]))
    assert res.idx[0, 0].tolist() == spec["selected"]


# ------------------------------------------------- exact rational brute force
def _rational_path(a, q_rows_per_head, W, kernel, kind, budget, reduce_order):
    """Exact fractions: keys ln(a_j), D = 1, scale 1, integer queries."""
    L = len(a)
    P = L - W
    sums = []
    for rows in q_rows_per_head:
        c = [Fraction(0)] * P
        for i, qi in enumerate(rows):
            e = [Fraction(a[j]) ** qi for j in range(P + i + 1)]
            tot = sum(e)
            for j in range(P):
                c[j] += e[j] / tot
        sums.append(c)
    r = (kernel - 1) // 2

    def pool(c):
        out = []
        for j in range(P):
            seg = c[max(0, j - r):min(P, j + r + 1)]
            out.append(max(seg) if kind == O.POOL_MAX else sum(seg) / kernel)
        return out

    if reduce_order == O.POOL_THEN_MEAN:
        pooled = [pool(c) for c in sums]
        score = [sum(p[j] for p in pooled) / len(pooled) for j in range(P)]
    else:
        score = pool([sum(c[j] for c in sums) / len(sums) for j in range(P)])
    if L <= budget:
        sel = list(range(L))
    else:
        order = sorted(range(P), key=lambda j: (-score[j], j))
        sel = sorted(order[:budget - W]) + list(range(P, L))
    return score, sel


@pytest.mark.parametrize("seed", range(12))
def test_rational_bruteforce(seed):
    rnd = random.Random(seed)
    W = rnd.randint(1, 4)
    L = rnd.randint(W + 1, 14)
    a = [rnd.randint(1, 5) for _ in range(L)]
    n_heads = rnd.randint(1, 3)
    q_rows = [[rnd.randint(-2, 3) for _ in range(W)] for _ in range(n_heads)]
    kernel = rnd.choice([1, 3, 5])
    kind = rnd.choice([O.POOL_MAX, O.POOL_AVG])
    order = rnd.choice([O.POOL_THEN_MEAN, O.MEAN_THEN_POOL])
    budget = rnd.randint(W, L + 1)
    exact, exact_sel = _rational_path(a, q_rows, W, kernel, kind, budget, order)
    keys = np.log(np.array(a, dtype=np.float64))[:, None]
    q_heads = [np.array(r, dtype=np.float64)[:, None] for r in q_rows]
    res = _layer(q_heads, keys, W, budget, kernel, kind, order, scale=1.0)
    P = L - W
    np.testing.assert_allclose(res.scores[0, :P], [float(x) for x in exact], rtol=1e-12, atol=0)
    got = [int(x) for x in res.idx[0, 0] if x >= 0]
    if got != exact_sel:
        # Only an exact rational tie may be broken differently after rounding.
        diff = set(got) ^ set(exact_sel)
        kept = [exact[j] for j in exact_sel if j < P]
        tau = min(kept) if kept else None
        assert tau is not None and all(exact[j] == tau for j in diff), (got, exact_sel)


# --------------------------------------------- scalar brute-force attention
def _scalar_causal_attention(q_all, k, scale):
    """Full causal attention, every query row, scalar loops and math.exp."""
    L, D = len(k), len(k[0])
    rows = []
    for t in range(L):
        logits = [scale * sum(q_all[t][d] * k[j][d] for d in range(D)) for j in range(t + 1)]
        m = max(logits)
        e = [math.exp(x - m) for x in logits]
        s = sum(e)
        rows.append([x / s for x in e] + [0.0] * (L - t - 1))
    return rows


@pytest.mark.parametrize("seed", range(6))
def test_window_attention_matches_scalar_bruteforce(seed):
    rng = np.random.default_rng(seed)
    L = int(rng.integers(8, 64))
    W = int(rng.integers(1, min(8, L) + 1))
    D = int(rng.integers(1, 9))
    scale = 1.0 / math.sqrt(D)
    q_all = rng.standard_normal((L, D))
    k = rng.standard_normal((L, D))
    full = _scalar_causal_attention(q_all.tolist(), k.tolist(), scale)
    a = O.row_softmax(O.window_logits(q_all[L - W:], k, scale))
    np.testing.assert_allclose(a, np.array(full[L - W:]), rtol=0, atol=1e-12)
    P = L - W
    c = O.window_column_sums(a, P)
    np.testing.assert_allclose(c, np.array(full[L - W:])[:, :P].sum(0), rtol=0, atol=1e-12)


def test_window_attention_matches_torch_softmax():
    rng = np.random.default_rng(7)
    L, W, D = 200, 16, 32
    q = rng.standard_normal((W, D))
    k = rng.standard_normal((L, D))
    scale = 0.3
    P = L - W
    logits = torch.from_numpy(q) @ torch.from_numpy(k).T * scale
    mask = torch.arange(L)[None, :] > (P + torch.arange(W))[:, None]
    ref = torch.softmax(logits.masked_fill(mask, float("-inf")), dim=-1).numpy()
    a = O.row_softmax(O.window_logits(q, k, scale))
    np.testing.assert_allclose(a, ref, rtol=1e-12, atol=1e-15)


def test_rows_sum_to_one_and_window_mass():
    rng = np.random.default_rng(3)
    L, W, D = 300, 24, 16
    q = 2.0 * rng.standard_normal((W, D))
    k = rng.standard_normal((L, D))
    a = O.row_softmax(O.window_logits(q, k, 0.25))
    np.testing.assert_allclose(a.sum(axis=1), np.ones(W), rtol=0, atol=1e-12)
    P = L - W
    c = O.window_column_sums(a, P)
    assert abs(c.sum() + a[:, P:].sum() - W) < 1e-11
    # causal: row i gives no mass to keys after position P + i
    for i in range(W):
        assert np.all(a[i, P + i + 1:] == 0.0)


def test_identical_keys_closed_form():
    """All keys equal: row i is uniform over P+i+1 keys, c[j] = sum_i 1/(P+i+1)."""
    rng = np.random.default_rng(5)
    L, W, D = 97, 9, 8
    k = np.tile(rng.standard_normal(D), (L, 1))
    q = rng.standard_normal((W, D))
    P = L - W
    c = O.window_column_sums(O.row_softmax(O.window_logits(q, k, 0.7)), P)
    expect = sum(1.0 / (P + i + 1) for i in range(W))
    np.testing.assert_allclose(c, np.full(P, expect), rtol=1e-13, atol=0)


# ------------------------------------------------------------------ pooling
@pytest.mark.parametrize("kernel", [1, 3, 5, 7, 9])
@pytest.mark.parametrize("P", [1, 2, 5, 40])
def test_pool_matches_torch(kernel, P):
    rng = np.random.default_rng(kernel * 100 + P)
    c = rng.random(P)
    r = (kernel - 1) // 2
    t = torch.from_numpy(c)[None, None]
    if r <= P:  # torch needs the padding within half the kernel and the input
        mx = F.max_pool1d(t, kernel, stride=1, padding=r)[0, 0].numpy()
        np.testing.assert_array_equal(O.pool1d(c, kernel, O.POOL_MAX), mx)
    av = F.avg_pool1d(t, kernel, stride=1, padding=r, count_include_pad=True)[0, 0].numpy()
    np.testing.assert_allclose(O.pool1d(c, kernel, O.POOL_AVG), av, rtol=1e-14, atol=0)


def test_pool_kernel_one_is_identity_and_even_rejected():
    c = np.random.default_rng(1).random(17)
    np.testing.assert_array_equal(O.pool1d(c, 1, O.POOL_MAX), c)
    np.testing.assert_array_equal(O.pool1d(c, 1, O.POOL_AVG), c)
    with pytest.raises(ValueError):
        O.pool1d(c, 4, O.POOL_MAX)


# ---------------------------------------------------------------- selection
@pytest.mark.parametrize("seed", range(10))
def test_select_matches_sorted_bruteforce(seed):
    rnd = random.Random(seed)
    W = rnd.randint(1, 8)
    L = rnd.randint(W, 200)
    budget = rnd.randint(W, L + 5)
    P = L - W
    # few distinct values, so ties are frequent
    score = np.array([rnd.choice([0.0, 0.25, 0.5, 1.0, 3.0]) for _ in range(P)])
    sel = O.select_tokens(score, L, W, budget)
    if L <= budget:
        assert sel.tolist() == list(range(L))
    else:
        best = sorted(range(P), key=lambda j: (-score[j], j))[:budget - W]
        assert sel.tolist() == sorted(best) + list(range(P, L))


def test_select_constant_scores_keeps_lowest_positions():
    L, W, B = 500, 16, 100
    sel = O.select_tokens(np.full(L - W, 0.5), L, W, B)
    assert sel.tolist() == list(range(B - W)) + list(range(L - W, L))


def test_select_invariants_and_nesting():
    rng = np.random.default_rng(11)
    L, W = 400, 8
    score = rng.random(L - W)
    prev = None
    for B in range(W, L + 3):
        sel = O.select_tokens(score, L, W, B)
        assert len(sel) == min(B, L)
        assert np.all(np.diff(sel) > 0)
        assert set(range(L - W, L)) <= set(sel.tolist())
        if prev is not None:
            assert set(prev.tolist()) <= set(sel.tolist())
        prev = sel
    with pytest.raises(ValueError):
        O.select_tokens(score, L, W, W - 1)


# ------------------------------------------------------------ metamorphic
def _rand_group(seed, n_heads=3, L=150, W=8, D=16):
    rng = np.random.default_rng(seed)
    return [rng.standard_normal((W, D)) for _ in range(n_heads)], rng.standard_normal((L, D))


def test_duplicate_and_permuted_srh_heads_leave_mean_unchanged():
    qs, k = _rand_group(21)
    base = O.group_scores(qs, k, 0.25, 5)
    np.testing.assert_allclose(O.group_scores(qs[::-1], k, 0.25, 5), base, rtol=1e-14)
    np.testing.assert_allclose(O.group_scores(qs + qs, k, 0.25, 5), base, rtol=1e-14)


def test_avg_pool_commutes_with_head_mean():
    qs, k = _rand_group(22)
    a = O.group_scores(qs, k, 0.25, 5, O.POOL_AVG, O.POOL_THEN_MEAN)
    b = O.group_scores(qs, k, 0.25, 5, O.POOL_AVG, O.MEAN_THEN_POOL)
    np.testing.assert_allclose(a, b, rtol=1e-13)
    one = O.group_scores(qs[:1], k, 0.25, 5, O.POOL_MAX, O.POOL_THEN_MEAN)
    np.testing.assert_allclose(one, O.group_scores(qs[:1], k, 0.25, 5, O.POOL_MAX,
                                                   O.MEAN_THEN_POOL), rtol=0)


def _small_layer(seed, batch=2, Hq=8, Hkv=2, D=16, W=8, lens=(90, 130)):
    rng = np.random.default_rng(seed)
    cu = np.concatenate([[0], np.cumsum(lens)])
    T = int(cu[-1])
    q = rng.standard_normal((batch, W, Hq, D))
    k = rng.standard_normal((T, Hkv, D))
    v = rng.standard_normal((T, Hkv, D))
    mask = np.array([1, 0, 1, 0, 0, 1, 0, 0], dtype=np.uint8)[:Hq]
    return q, k, v, cu, mask


def test_unrelated_inputs_do_not_change_selection():
    q, k, v, cu, mask = _small_layer(31)
    base = O.compress_layer(q, k, v, cu, mask, 40, 5)
    rng = np.random.default_rng(99)
    q2 = q.copy()
    q2[:, :, mask == 0, :] = rng.standard_normal(q2[:, :, mask == 0, :].shape)
    r = O.compress_layer(q2, k, v, cu, mask, 40, 5)
    np.testing.assert_array_equal(r.idx, base.idx)
    v2 = rng.standard_normal(v.shape)
    np.testing.assert_array_equal(O.compress_layer(q, k, v2, cu, mask, 40, 5).idx, base.idx)
    k2 = k.copy()
    k2[:, 1, :] = rng.standard_normal(k2[:, 1, :].shape)   # group 1 changes, group 0 must not
    r = O.compress_layer(q, k2, v, cu, mask, 40, 5)
    np.testing.assert_array_equal(r.idx[:, 0], base.idx[:, 0])


def test_ragged_batch_equals_sequences_alone():
    q, k, v, cu, mask = _small_layer(41)
    both = O.compress_layer(q, k, v, cu, mask, 50, 7)
    for b in range(2):
        s0, s1 = cu[b], cu[b + 1]
        one = O.compress_layer(q[b:b + 1], k[s0:s1], v[s0:s1], np.array([0, s1 - s0]), mask, 50, 7)
        np.testing.assert_array_equal(one.idx[0], both.idx[b])
        np.testing.assert_array_equal(one.scores, both.scores[:, s0:s1])


def test_all_heads_mask_is_snapkv_gqa():
    """SRH mask = every head of a group gives SnapKV's group-averaged selection,
    computed here with batched torch ops over all heads at once."""
    q, k, v, cu, _ = _small_layer(51, batch=1, lens=(160,))
    Hq, Hkv, W, D = 8, 2, 8, 16
    G = Hq // Hkv
    mask = np.ones(Hq, dtype=np.uint8)
    res = O.compress_layer(q, k, v, cu, mask, 48, 5)
    L = 160
    P = L - W
    qt = torch.from_numpy(q[0]).permute(1, 0, 2)                    # [Hq, W, D]
    kt = torch.from_numpy(k).permute(1, 0, 2).repeat_interleave(G, 0)  # [Hq, L, D]
    att = torch.matmul(qt, kt.transpose(1, 2).contiguous()) / math.sqrt(D)
    causal = torch.arange(L)[None, :] > (P + torch.arange(W))[:, None]
    att = torch.softmax(att.masked_fill(causal, float("-inf")), dim=-1)
    vote = att[:, :, :P].sum(1)                                      # [Hq, P]
    pooled = F.max_pool1d(vote[:, None], 5, stride=1, padding=2)[:, 0]
    group = pooled.view(Hkv, G, P).mean(1)                           # [Hkv, P]
    np.testing.assert_allclose(res.scores[:, :P], group.numpy(), rtol=1e-12)
    for g in range(Hkv):
        top = torch.topk(group[g], 48 - W).indices.sort().values.tolist()
        assert res.idx[0, g].tolist() == top + list(range(P, L))


def test_gather_is_bit_copy_and_padding():
    q, k, v, cu, mask = _small_layer(61)
    kb = k.astype(np.float32).view(np.uint32)   # raw bits, copied verbatim
    vb = v.astype(np.float32).view(np.uint32)
    res = O.compress_layer(q, kb, vb, cu, mask, 100, 3, k_values=k.astype(np.float32))
    for b in range(2):
        L = cu[b + 1] - cu[b]
        n = min(100, L)
        for g in range(2):
            sel = res.idx[b, g, :n]
            np.testing.assert_array_equal(res.k_out[b, g, :n], kb[cu[b] + sel, g])
            np.testing.assert_array_equal(res.v_out[b, g, :n], vb[cu[b] + sel, g])
            assert np.all(res.idx[b, g, n:] == -1)
            assert np.all(res.k_out[b, g, n:] == 0)


def test_group_without_srh_is_rejected():
    q, k, v, cu, _ = _small_layer(71)
    mask = np.array([1, 0, 0, 0, 0, 0, 0, 0], dtype=np.uint8)
    with pytest.raises(ValueError):
        O.compress_layer(q, k, v, cu, mask, 40, 5)
