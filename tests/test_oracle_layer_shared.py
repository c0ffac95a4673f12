"""Pins of the oracle's layer-shared index set (section 3.3: every head of a
layer keeps the tokens chosen by the average of the layer's pooled SRH
vectors, each SRH attending to its own KV group's keys).

The reference computation below is independent of the oracle's code: all
heads at once with batched torch ops (attention via matmul + softmax, the
window sum, F.max_pool1d / F.avg_pool1d, a mean over the SRH axis and
torch.topk with the lowest-index tie rule written out)."""
import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle as O


def _layer(seed, batch=1, Hq=8, Hkv=2, D=16, W=8, lens=(150,)):
    rng = np.random.default_rng(seed)
    cu = np.concatenate([[0], np.cumsum(lens)])
    T = int(cu[-1])
    q = rng.standard_normal((batch, W, Hq, D))
    k = rng.standard_normal((T, Hkv, D))
    v = rng.standard_normal((T, Hkv, D))
    return q, k, v, cu


def _torch_layer_score(q, k, mask, W, kernel, pool):
    """Layer score of one sequence: q [W, Hq, D], k [L, Hkv, D]."""
    Hq, Hkv = q.shape[1], k.shape[1]
    G = Hq // Hkv
    L, D = k.shape[0], k.shape[2]
    P = L - W
    qt = torch.from_numpy(q).permute(1, 0, 2)                            # [Hq, W, D]
    kt = torch.from_numpy(k).permute(1, 0, 2).repeat_interleave(G, 0)    # [Hq, L, D]
    att = torch.matmul(qt, kt.transpose(1, 2).contiguous()) / math.sqrt(D)
    causal = torch.arange(L)[None, :] > (P + torch.arange(W))[:, None]
    att = torch.softmax(att.masked_fill(causal, float("-inf")), dim=-1)
    vote = att[:, :, :P].sum(1)                                         # [Hq, P]
    r = (kernel - 1) // 2
    if pool == O.POOL_MAX:
        pooled = F.max_pool1d(vote[:, None], kernel, stride=1, padding=r)[:, 0]
    else:
        pooled = F.avg_pool1d(vote[:, None], kernel, stride=1, padding=r,
                              count_include_pad=True)[:, 0]
    sel = torch.from_numpy(np.nonzero(mask)[0])
    return pooled[sel].mean(0)                                           # [P]


def _torch_select(score, L, W, budget):
    P = L - W
    if L <= budget:
        return list(range(L))
    # lowest index first among equal scores: sort by (-score, index)
    order = sorted(range(P), key=lambda j: (-float(score[j]), j))
    return sorted(order[:budget - W]) + list(range(P, L))


@pytest.mark.parametrize("seed,pool,mask", [
    (0, O.POOL_MAX, [1, 0, 0, 0, 1, 1, 1, 0]),     # groups with 1 and 3 SRHs
    (1, O.POOL_AVG, [0, 1, 0, 1, 0, 0, 1, 0]),
    (2, O.POOL_MAX, [1, 1, 1, 1, 0, 0, 0, 0]),     # group 1 has no SRH
])
def test_layer_shared_matches_batched_torch(seed, pool, mask):
    q, k, v, cu = _layer(seed, batch=2, lens=(150, 97))
    mask = np.array(mask, dtype=np.uint8)
    W, kernel, budget = 8, 5, 40
    res = O.compress_layer(q, k, v, cu, mask, budget, kernel, pool, index_mode=O.LAYER_SHARED)
    for b in range(2):
        s0, s1 = int(cu[b]), int(cu[b + 1])
        L = s1 - s0
        P = L - W
        want = _torch_layer_score(q[b], k[s0:s1], mask, W, kernel, pool).numpy()
        for g in range(2):
            np.testing.assert_allclose(res.scores[g, s0:s0 + P], want, rtol=1e-12, atol=0)
            assert np.all(np.isinf(res.scores[g, s0 + P:s1]))
            sel = _torch_select(want, L, W, budget)
            assert res.idx[b, g, :len(sel)].tolist() == sel
            np.testing.assert_array_equal(res.k_out[b, g, :len(sel)], k[s0 + np.array(sel), g])
            np.testing.assert_array_equal(res.v_out[b, g, :len(sel)], v[s0 + np.array(sel), g])


def test_single_group_layer_shared_equals_per_group():
    q, k, v, cu = _layer(3, Hq=4, Hkv=1)
    mask = np.array([1, 0, 1, 1], dtype=np.uint8)
    a = O.compress_layer(q, k, v, cu, mask, 48, 7)
    b = O.compress_layer(q, k, v, cu, mask, 48, 7, index_mode=O.LAYER_SHARED)
    np.testing.assert_array_equal(a.idx, b.idx)
    np.testing.assert_allclose(a.scores, b.scores, rtol=1e-14)


def test_layer_score_weights_heads_not_groups():
    """The layer score is the mean over SRHs, so a group's per-group score
    counts with its number of SRHs."""
    q, k, v, cu = _layer(4)
    mask = np.array([1, 0, 0, 0, 1, 1, 1, 0], dtype=np.uint8)    # 1 and 3 SRHs
    per = O.compress_layer(q, k, v, cu, mask, 40, 5)
    lay = O.compress_layer(q, k, v, cu, mask, 40, 5, index_mode=O.LAYER_SHARED)
    P = 150 - 8
    np.testing.assert_allclose(lay.scores[0, :P], (per.scores[0, :P] + 3 * per.scores[1, :P]) / 4,
                               rtol=1e-12)
    assert not np.allclose(lay.scores[0, :P], (per.scores[0, :P] + per.scores[1, :P]) / 2)


def test_keys_of_a_group_without_srh_do_not_change_the_selection():
    q, k, v, cu = _layer(5)
    mask = np.array([0, 1, 1, 0, 0, 0, 0, 0], dtype=np.uint8)    # group 1: no SRH
    base = O.compress_layer(q, k, v, cu, mask, 40, 5, index_mode=O.LAYER_SHARED)
    k2 = k.copy()
    k2[:, 1, :] = np.random.default_rng(6).standard_normal(k2[:, 1, :].shape)
    r = O.compress_layer(q, k2, v, cu, mask, 40, 5, index_mode=O.LAYER_SHARED)
    np.testing.assert_array_equal(r.idx, base.idx)
    np.testing.assert_array_equal(r.k_out[:, 1], k2[r.idx[0, 1]][None, :, 1])
    np.testing.assert_array_equal(base.idx[:, 0], base.idx[:, 1])


def test_group_order_does_not_matter():
    q, k, v, cu = _layer(7)
    mask = np.array([1, 0, 1, 0, 0, 1, 0, 0], dtype=np.uint8)
    base = O.compress_layer(q, k, v, cu, mask, 36, 5, index_mode=O.LAYER_SHARED)
    qs = np.concatenate([q[:, :, 4:], q[:, :, :4]], axis=2)       # swap the two groups
    ks = k[:, ::-1].copy()
    vs = v[:, ::-1].copy()
    ms = np.concatenate([mask[4:], mask[:4]])
    r = O.compress_layer(qs, ks, vs, cu, ms, 36, 5, index_mode=O.LAYER_SHARED)
    np.testing.assert_array_equal(r.idx[:, 0], base.idx[:, 0])
    np.testing.assert_allclose(r.scores[0], base.scores[0], rtol=1e-13)


def test_layer_shared_rejections():
    q, k, v, cu = _layer(8)
    with pytest.raises(ValueError):
        O.compress_layer(q, k, v, cu, np.zeros(8, dtype=np.uint8), 40, 5,
                         index_mode=O.LAYER_SHARED)
    with pytest.raises(ValueError):
        O.compress_layer(q, k, v, cu, np.ones(8, dtype=np.uint8), 40, 5,
                         reduce_order=O.MEAN_THEN_POOL, index_mode=O.LAYER_SHARED)
