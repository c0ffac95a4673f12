"""Pins of the oracle's per-group budgets (compress_layer_heads): with equal
budgets it is compress_layer laid out group after group; each group's result
depends on its own budget only and equals the fixed-budget selection at that
budget; the selection nests as a group's budget grows."""
import numpy as np

import oracle as O


def _layer(seed, lens=(300, 170), Hq=8, Hkv=4, D=16, W=8):
    rng = np.random.default_rng(seed)
    cu = np.concatenate([[0], np.cumsum(lens)])
    q = rng.standard_normal((len(lens), W, Hq, D))
    k = rng.standard_normal((int(cu[-1]), Hkv, D))
    v = rng.standard_normal((int(cu[-1]), Hkv, D))
    mask = np.zeros(Hq, dtype=np.uint8)
    mask[::2] = 1
    return q, k, v, cu, mask


def test_equal_budgets_are_the_fixed_budget_layout():
    q, k, v, cu, mask = _layer(1)
    ref = O.compress_layer(q, k, v, cu, mask, 40, 5)
    got = O.compress_layer_heads(q, k, v, cu, mask, [40] * 4, 5)
    assert np.array_equal(got.idx, ref.idx.reshape(2, -1))
    assert np.array_equal(got.k_out, ref.k_out.reshape(2, 4 * 40, -1))
    assert np.array_equal(got.scores, ref.scores)


def test_each_group_follows_its_own_budget():
    q, k, v, cu, mask = _layer(2)
    budgets = [8, 60, 171, 33]            # W, mid, above the shorter length, mid
    got = O.compress_layer_heads(q, k, v, cu, mask, budgets, 3, pool_type=O.POOL_AVG)
    off = np.concatenate([[0], np.cumsum(budgets)])
    for g, B in enumerate(budgets):
        ref = O.compress_layer(q, k, v, cu, mask, B, 3, pool_type=O.POOL_AVG)
        assert np.array_equal(got.idx[:, off[g]:off[g + 1]], ref.idx[:, g])
        assert np.array_equal(got.v_out[:, off[g]:off[g + 1]], ref.v_out[:, g])
    # changing one group's budget leaves the other groups' slices unchanged
    budgets2 = [8, 61, 171, 33]
    got2 = O.compress_layer_heads(q, k, v, cu, mask, budgets2, 3, pool_type=O.POOL_AVG)
    off2 = np.concatenate([[0], np.cumsum(budgets2)])
    for g in (0, 2, 3):
        assert np.array_equal(got.idx[:, off[g]:off[g + 1]], got2.idx[:, off2[g]:off2[g + 1]])


def test_selection_nests_as_the_budget_grows():
    q, k, v, cu, mask = _layer(3)
    small = O.compress_layer_heads(q, k, v, cu, mask, [20, 20, 20, 20], 5)
    big = O.compress_layer_heads(q, k, v, cu, mask, [20, 45, 20, 20], 5)
    for b in range(2):
        s = set(small.idx[b, 20:40].tolist()) - {-1}
        t = set(big.idx[b, 20:65].tolist()) - {-1}
        assert s <= t
