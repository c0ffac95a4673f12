"""Plant plausible mistakes in the offline oracle (CPU only) and check that
the pins of tests/test_oracle_offline.py reject every one of them."""
import math

import numpy as np
import pytest

import oracle.offline_oracle as M
from tests import test_oracle_offline as pins


def _srh_all_steps(attn, gen_tokens, ctx_tokens, spans):
    S, N, H, L = attn.shape
    out = np.zeros(H)
    for s in range(S):
        a0, n = int(spans[s, 0]), int(spans[s, 1])
        out += attn[s, :, :, a0:a0 + n].sum(axis=(0, 2))     # ignores whether y_t is an answer token
    return out


def _srh_span_off_by_one(attn, gen_tokens, ctx_tokens, spans):
    sp = np.array(spans).copy()
    sp[:, 1] += 1
    return _orig["srh_scores"](attn, gen_tokens, ctx_tokens, np.minimum(sp, attn.shape[3]))


def _srh_peak_not_mass(attn, gen_tokens, ctx_tokens, spans):
    S, N, H, L = attn.shape
    out = np.zeros(H)
    for s in range(S):
        a0, n = int(spans[s, 0]), int(spans[s, 1])
        hit = M.answer_hits(gen_tokens[s], ctx_tokens[s], a0, n)
        for t in range(N):
            if hit[t]:
                out += attn[s, t, :, a0:a0 + n].max(axis=1)   # top weight, not the span mass
    return out


def _select_high_index_ties(scores, n_layers, top_k):
    sc = np.asarray(scores, dtype=np.float64).reshape(n_layers, -1)
    mask = np.zeros(sc.shape, dtype=np.uint8)
    for l in range(n_layers):
        for h in sorted(range(sc.shape[1]), key=lambda h: (-sc[l, h], -h))[:top_k]:
            mask[l, h] = 1
    return mask


def _attn_unscaled(q, k, v, scale):
    return _orig["decode_attention"](q, k, v, 1.0)


def _attn_wrong_group_map(q, k, v, scale):
    Hq, Hkv = q.shape[0], k.shape[1]
    out = np.zeros(q.shape)
    for h in range(Hq):
        g = h % Hkv                                           # interleaved instead of contiguous
        z = scale * (k[:, g, :] @ q[h])
        w = np.exp(z - z.max())
        out[h] = (w / w.sum()) @ v[:, g, :]
    return out


def _error_without_projection(q_dec, k, v, cu, idx, w_o, eps=1e-6, scale=None):
    return _orig["layer_error"](q_dec, k, v, cu, idx, np.eye(w_o.shape[1]), eps, scale)


def _error_relative_to_compressed(q_dec, k, v, cu, idx, w_o, eps=1e-6, scale=None):
    batch, T, Hq, D = q_dec.shape
    scale = 1 / math.sqrt(D) if not scale else scale
    e = 0.0
    for b in range(batch):
        kf, vf = k[cu[b]:cu[b + 1]], v[cu[b]:cu[b + 1]]
        for t in range(T):
            a_full = M.decode_attention(q_dec[b, t], kf, vf, scale)
            G = Hq // k.shape[1]
            a_comp = np.zeros_like(a_full)
            for g in range(k.shape[1]):
                keep = idx[b, g][idx[b, g] >= 0]
                a_comp[g * G:(g + 1) * G] = M.decode_attention(
                    q_dec[b, t, g * G:(g + 1) * G], kf[keep][:, g:g + 1], vf[keep][:, g:g + 1], scale)
            d = np.linalg.norm(w_o @ (a_full - a_comp).reshape(-1))
            e += d / (np.linalg.norm(w_o @ a_comp.reshape(-1)) + eps)   # wrong reference
    return e


def _budget_clamp_only(e_norm, total, m, M_):
    n = len(e_norm)
    share = (total - n * m) * np.asarray(e_norm) / np.sum(e_norm)
    out = np.minimum(m + np.floor(share).astype(np.int64), M_)          # excess is lost
    left = total - out.sum()
    for i in np.argsort(-(share - np.floor(share)), kind="stable")[:max(left, 0)]:
        out[i] += 1
    return out


def _budget_share_of_total(e_norm, total, m, M_):
    n = len(e_norm)
    share = total * np.asarray(e_norm)                                  # ignores the minimum
    out = np.clip(np.floor(share).astype(np.int64), m, M_)
    return out


def _budget_remainder_to_first(e_norm, total, m, M_):
    out = _orig["allocate_budgets"](e_norm, total, m, M_)
    e = np.asarray(e_norm)
    free = np.flatnonzero(out < M_)
    rest = total - out[out >= M_].sum() - m * len(free)
    share = rest * e[free] / e[free].sum()
    fl = m + np.floor(share).astype(np.int64)
    out[free] = fl
    left = total - out.sum()
    out[free[:left]] += 1                                               # lowest layers, not largest parts
    return out


def _normalise_by_max(e):
    e = np.asarray(e, dtype=np.float64)
    return e / e.max()                                                  # largest error -> 1


def _normalise_identity(e):
    return np.asarray(e, dtype=np.float64)                              # no normalisation


_orig = {n: getattr(M, n) for n in ("srh_scores", "select_srh", "decode_attention", "layer_error",
                                    "allocate_budgets", "normalize_errors")}

MUTANTS = {
    "every step counted": ("srh_scores", _srh_all_steps),
    "span one position too long": ("srh_scores", _srh_span_off_by_one),
    "peak weight instead of span mass": ("srh_scores", _srh_peak_not_mass),
    "head ties to the higher index": ("select_srh", _select_high_index_ties),
    "attention scale dropped": ("decode_attention", _attn_unscaled),
    "interleaved GQA map": ("decode_attention", _attn_wrong_group_map),
    "no output projection": ("layer_error", _error_without_projection),
    "error relative to the compressed output": ("layer_error", _error_relative_to_compressed),
    "cap excess dropped": ("allocate_budgets", _budget_clamp_only),
    "shares of the total, not of the rest": ("allocate_budgets", _budget_share_of_total),
    "rounding units to the lowest layers": ("allocate_budgets", _budget_remainder_to_first),
    "errors normalised by their maximum": ("normalize_errors", _normalise_by_max),
    "errors not normalised": ("normalize_errors", _normalise_identity),
}

PINS = [
    pins.test_srh_score_hand_worked_example,
    pins.test_srh_score_equals_masked_einsum,
    pins.test_srh_score_closed_forms,
    pins.test_srh_score_is_linear_and_ignores_other_positions,
    pins.test_select_srh_ranks_each_layer_with_lowest_index_ties,
    pins.test_layer_error_matches_batched_torch,
    pins.test_layer_error_closed_forms,
    pins.test_layer_error_invariants,
    pins.test_budget_hand_worked_example,
    pins.test_budget_closed_forms,
    lambda: [pins.test_normalised_errors_are_shares(s) for s in range(4)],
    lambda: [pins.test_budget_invariants(s) for s in range(6)],
]


@pytest.mark.parametrize("label", sorted(MUTANTS))
def test_pins_reject_offline_mutant(label, monkeypatch):
    name, fn = MUTANTS[label]
    monkeypatch.setattr(M, name, fn)
    monkeypatch.setattr(pins.OO, name, fn)
    caught = False
    for pin in PINS:
        try:
            pin()
        except (AssertionError, ValueError, IndexError):
            caught = True
            break
    assert caught, f"no pin rejects the mutant: {label}"


def test_unmutated_offline_oracle_passes_all_pins():
    for pin in PINS:
        pin()
