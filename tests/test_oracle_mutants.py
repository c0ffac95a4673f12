"""Plant plausible mistakes in the oracle (CPU only) and check that the pins
catch every one of them.  A mutant that no pin rejects would mean the pins do
not really tie the oracle down."""
import numpy as np
import pytest

import oracle as O
import oracle.compresskv_oracle as M
from tests import test_oracle_layer_shared as lpins
from tests import test_oracle_pins as pins
from tests import test_workloads as wtests


def _logits_no_window_in_denominator(q_head, k_seq, scale):
    z = _orig["window_logits"](q_head, k_seq, scale)
    z[:, k_seq.shape[0] - q_head.shape[0]:] = -np.inf   # forgets the window keys
    return z


def _logits_causal_off_by_one(q_head, k_seq, scale):
    W, L = q_head.shape[0], k_seq.shape[0]
    z = scale * (q_head @ k_seq.T)
    for i in range(W):
        z[i, L - W + i:] = -np.inf                       # drops the diagonal
    return z


def _logits_unscaled(q_head, k_seq, scale):
    return _orig["window_logits"](q_head, k_seq, 1.0)


def _colsum_mean(a, P):
    return np.mean(a[:, :P], axis=0)


def _colsum_with_window(a, P):
    return np.sum(a, axis=0)[:P] + np.sum(a[:, P:]) / max(P, 1)


def _pool_avg_exclude_pad(c, kernel, kind):
    if kind == O.POOL_MAX:
        return _orig["pool1d"](c, kernel, kind)
    P, r = c.shape[0], (kernel - 1) // 2
    return np.array([np.mean(c[max(0, j - r):min(P, j + r + 1)]) for j in range(P)])


def _pool_off_center(c, kernel, kind):
    P = c.shape[0]
    out = np.empty(P)
    for j in range(P):
        seg = c[j:min(P, j + kernel)]
        out[j] = seg.max() if kind == O.POOL_MAX else seg.sum() / kernel
    return out


def _select_highest_index_ties(score, L, window, budget):
    if L <= budget:
        return np.arange(L)
    P = L - window
    order = np.lexsort((-np.arange(P), -score))
    return np.concatenate([np.sort(order[:budget - window]), np.arange(P, L)])


def _select_budget_excludes_window(score, L, window, budget):
    if L <= budget + window:
        return np.arange(L)
    P = L - window
    order = np.lexsort((np.arange(P), -score))
    return np.concatenate([np.sort(order[:budget]), np.arange(P, L)])


def _select_smallest(score, L, window, budget):
    if L <= budget:
        return np.arange(L)
    P = L - window
    order = np.lexsort((np.arange(P), score))
    return np.concatenate([np.sort(order[:budget - window]), np.arange(P, L)])


def _group_scores_sum_heads(q_heads, k_seq, scale, pool_kernel, pool_type=0, reduce_order=0):
    s = _orig["group_scores"](q_heads, k_seq, scale, pool_kernel, pool_type, reduce_order)
    return s * len(q_heads) if len(q_heads) > 1 else s + 0.0


def _group_scores_wrong_order(q_heads, k_seq, scale, pool_kernel, pool_type=0, reduce_order=0):
    return _orig["group_scores"](q_heads, k_seq, scale, pool_kernel, pool_type, 1 - reduce_order)


def _layer_scores_first_group_keys(q_and_keys, scale, pool_kernel, pool_type=0):
    k0 = q_and_keys[0][1]                                # every SRH reads group 0's keys
    return _orig["layer_scores"]([(q, k0) for q, _ in q_and_keys], scale, pool_kernel, pool_type)


def _layer_scores_sum(q_and_keys, scale, pool_kernel, pool_type=0):
    return _orig["layer_scores"](q_and_keys, scale, pool_kernel, pool_type) * len(q_and_keys)


_orig = {name: getattr(M, name) for name in
         ("window_logits", "window_column_sums", "pool1d", "select_tokens", "group_scores",
          "layer_scores")}

MUTANTS = {
    "window keys left out of the softmax": ("window_logits", _logits_no_window_in_denominator),
    "causal mask off by one": ("window_logits", _logits_causal_off_by_one),
    "softmax scale dropped": ("window_logits", _logits_unscaled),
    "mean instead of sum over window": ("window_column_sums", _colsum_mean),
    "window mass leaks into prefix sums": ("window_column_sums", _colsum_with_window),
    "avg pooling without zero padding": ("pool1d", _pool_avg_exclude_pad),
    "pooling window not centred": ("pool1d", _pool_off_center),
    "ties to the highest index": ("select_tokens", _select_highest_index_ties),
    "budget does not count the window": ("select_tokens", _select_budget_excludes_window),
    "keeps the lowest scores": ("select_tokens", _select_smallest),
    "sum over SRHs instead of mean": ("group_scores", _group_scores_sum_heads),
    "pool and head mean swapped": ("group_scores", _group_scores_wrong_order),
    "layer SRHs read one group's keys": ("layer_scores", _layer_scores_first_group_keys),
    "sum over the layer's SRHs": ("layer_scores", _layer_scores_sum),
}

PINS = [
    lambda: [pins.test_hand_worked_examples(n) for n in
             ("worked_max3.txt", "worked_avg3.txt", "worked_two_heads.txt")],
    lambda: [pins.test_rational_bruteforce(s) for s in range(12)],
    lambda: [pins.test_window_attention_matches_scalar_bruteforce(s) for s in range(3)],
    pins.test_window_attention_matches_torch_softmax,
    pins.test_identical_keys_closed_form,
    lambda: pins.test_pool_matches_torch(5, 40),
    lambda: [pins.test_select_matches_sorted_bruteforce(s) for s in range(10)],
    pins.test_select_constant_scores_keeps_lowest_positions,
    pins.test_all_heads_mask_is_snapkv_gqa,
    lambda: wtests.test_needles_retained_by_oracle_on_tiny(0),
    lambda: lpins.test_layer_shared_matches_batched_torch(0, O.POOL_MAX,
                                                          [1, 0, 0, 0, 1, 1, 1, 0]),
    lpins.test_layer_score_weights_heads_not_groups,
]


@pytest.mark.parametrize("label", sorted(MUTANTS))
def test_pins_reject_mutant(label, monkeypatch):
    name, fn = MUTANTS[label]
    monkeypatch.setattr(M, name, fn)
    monkeypatch.setattr(O, name, fn)
    caught = False
    for pin in PINS:
        try:
            pin()
        except (AssertionError, ValueError, IndexError):
            caught = True
            break
    assert caught, f"no pin rejects the mutant: {label}"


def test_unmutated_oracle_passes_all_pins():
    for pin in PINS:
        pin()
