"""Plain, slow, fp64 CPU oracle of CompressKV's offline analyses.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or call this module.  The
product path never touches it, and this module imports nothing from the
product package.

What it computes:

  * the Semantic Retrieval Head score of every attention head (section 3.2,
    equation 1): over the decoding steps of calibration samples, the
    attention mass a head puts on the answer span, counted at the steps whose
    generated token belongs to the answer;
  * the SRH set of every layer: its top-k heads by that score (section 3.3);
  * the eviction error of a layer (section 3.4, equations 2-4): over decoding
    steps, the Frobenius norm of the difference between the attention block's
    output (after the output projection) with the compressed and with the full
    KV cache, relative to the full-cache output;
  * the layer budgets: a minimum m per layer, the rest of the total in
    proportion to the normalised errors, each layer capped at M (section 3.4
    and section 4, "Implementation Details").

Readings of points the paper leaves open (restated where used, and listed in
the repository's design notes):

  * "the generated token belongs to the answer span" compares token ids: step
    t counts when y_t equals the token id at some position of the span;
  * ties in the top-k head ranking go to the lower head index;
  * a decoding step's query attends to the cached prompt only (full: every
    position, compressed: the kept positions); the decoding steps' own new
    tokens are left out of both caches, so the two outputs differ only by the
    eviction;
  * query head h reads KV group h // (Hq // Hkv); the heads' outputs are
    concatenated head-major before the output projection;
  * budgets are integers: the proportional shares of the remainder are
    floored, layers at the cap M are frozen and their excess is shared again
    among the others, and the last units left by flooring go one each to the
    largest fractional parts (ties: lower layer index).

Parity status: every function is pinned by tests/test_oracle_offline.py
against closed forms, brute force, invariants and hand-worked examples; the
paper prints no worked numbers for these analyses.
"""
from __future__ import annotations

import math

import numpy as np


# --------------------------------------------------------------------------
# Equation 1: the SRH score.
# --------------------------------------------------------------------------
def answer_hits(gen_tokens: np.ndarray, ctx_tokens: np.ndarray, span_start: int,
                span_len: int) -> np.ndarray:
    """1 where the generated token of step t is one of the answer's tokens.

    gen_tokens: [N] token ids generated at the N decoding steps.
    ctx_tokens: [L] token ids of the context; the answer span is
    ctx_tokens[span_start : span_start + span_len].
    """
    answer = set(int(x) for x in ctx_tokens[span_start:span_start + span_len])
    return np.array([1 if int(y) in answer else 0 for y in gen_tokens], dtype=np.int64)


def srh_scores(attn: np.ndarray, gen_tokens: np.ndarray, ctx_tokens: np.ndarray,
               spans: np.ndarray) -> np.ndarray:
    """S(h) = sum over samples and steps t with y_t in the answer of the
    attention weight head h puts on the answer span.

    attn: [S, N, H, L] attention weights of the H heads at the N decoding steps
          of each of S samples over the L context positions.
    gen_tokens: [S, N]; ctx_tokens: [S, L]; spans: [S, 2] (start, length).
    Returns [H] in float64.
    """
    S, N, H, L = attn.shape
    out = np.zeros(H, dtype=np.float64)
    for s in range(S):
        a0, n = int(spans[s, 0]), int(spans[s, 1])
        hit = answer_hits(gen_tokens[s], ctx_tokens[s], a0, n)
        for t in range(N):
            if hit[t]:
                out += np.asarray(attn[s, t, :, a0:a0 + n], dtype=np.float64).sum(axis=1)
    return out


def select_srh(scores: np.ndarray, n_layers: int, top_k: int) -> np.ndarray:
    """SRH mask [n_layers, heads per layer]: each layer's top_k heads by score
    (ties: lower head index).  scores: [n_layers * heads per layer]."""
    sc = np.asarray(scores, dtype=np.float64).reshape(n_layers, -1)
    mask = np.zeros(sc.shape, dtype=np.uint8)
    for l in range(n_layers):
        order = sorted(range(sc.shape[1]), key=lambda h: (-sc[l, h], h))
        for h in order[:top_k]:
            mask[l, h] = 1
    return mask


# --------------------------------------------------------------------------
# Equations 2-4: the eviction error of a layer.
# --------------------------------------------------------------------------
def decode_attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, scale: float) -> np.ndarray:
    """Softmax attention of one decoding query per head over a cache.

    q: [Hq, D]; k, v: [n, Hkv, D] (the cached positions of one sequence).
    Head h reads group h // (Hq // Hkv).  Returns [Hq, D] in float64.
    """
    Hq, D = q.shape
    Hkv = k.shape[1]
    G = Hq // Hkv
    out = np.zeros((Hq, D), dtype=np.float64)
    for h in range(Hq):
        g = h // G
        z = scale * (np.asarray(k[:, g, :], dtype=np.float64) @ np.asarray(q[h], dtype=np.float64))
        w = np.exp(z - z.max())
        w /= w.sum()
        out[h] = w @ np.asarray(v[:, g, :], dtype=np.float64)
    return out


def layer_error(q_dec: np.ndarray, k: np.ndarray, v: np.ndarray, cu_seqlens: np.ndarray,
                idx: np.ndarray, w_o: np.ndarray, eps: float = 1e-6,
                scale: float | None = None) -> float:
    """e = sum over sequences b and decoding steps t of
    ||W_O (A_full - A_comp)||_F / (||W_O A_full||_F + eps).

    q_dec: [batch, T, Hq, D] decoding queries; k, v: [T_total, Hkv, D] packed
    full caches (cu_seqlens); idx: [batch, Hkv, B] kept positions per group
    (-1 = none), as the eviction path writes them; w_o: [d_model, Hq*D].
    """
    batch, T, Hq, D = q_dec.shape
    Hkv = k.shape[1]
    if scale is None or scale <= 0:
        scale = 1.0 / math.sqrt(D)
    W = np.asarray(w_o, dtype=np.float64)
    e = 0.0
    for b in range(batch):
        s0, s1 = int(cu_seqlens[b]), int(cu_seqlens[b + 1])
        kf = np.asarray(k[s0:s1], dtype=np.float64)
        vf = np.asarray(v[s0:s1], dtype=np.float64)
        for t in range(T):
            a_full = decode_attention(q_dec[b, t], kf, vf, scale)
            a_comp = np.zeros_like(a_full)
            G = Hq // Hkv
            for g in range(Hkv):
                keep = idx[b, g][idx[b, g] >= 0]
                part = decode_attention(q_dec[b, t, g * G:(g + 1) * G], kf[keep][:, g:g + 1, :],
                                        vf[keep][:, g:g + 1, :], scale)
                a_comp[g * G:(g + 1) * G] = part
            o_full = W @ a_full.reshape(-1)
            o_diff = W @ (a_full - a_comp).reshape(-1)
            e += np.linalg.norm(o_diff) / (np.linalg.norm(o_full) + eps)
    return float(e)


def normalize_errors(e: np.ndarray) -> np.ndarray:
    """e~(l) = e(l) / sum_k e(k)."""
    e = np.asarray(e, dtype=np.float64)
    return e / e.sum()


def allocate_budgets(e_norm: np.ndarray, total: int, m: int, M: int) -> np.ndarray:
    """Integer layer budgets in [m, M] summing to `total`: m each, the rest in
    proportion to e_norm, layers that would pass M held at M and their excess
    shared again among the others; units left by flooring go to the largest
    fractional parts (ties: lower layer index)."""
    e = np.asarray(e_norm, dtype=np.float64)
    n = e.shape[0]
    if not (n * m <= total <= n * M):
        raise ValueError("total must lie in [n*m, n*M]")
    budget = np.full(n, m, dtype=np.int64)
    capped = np.zeros(n, dtype=bool)
    while True:
        rest = total - budget[capped].sum() - m * int((~capped).sum())
        weights = np.where(capped, 0.0, e)
        wsum = weights.sum()
        share = np.zeros(n) if wsum == 0 else rest * weights / wsum
        if wsum == 0:   # every free layer has zero error: split the rest evenly
            free = np.flatnonzero(~capped)
            share[free] = rest / len(free)
        over = (~capped) & (m + share > M)
        if not over.any():
            break
        budget[over] = M
        capped |= over
    floor = np.floor(share).astype(np.int64)
    out = budget.copy()
    out[~capped] = m + floor[~capped]
    left = total - int(out.sum())
    frac = share - floor
    order = sorted(np.flatnonzero(~capped).tolist(), key=lambda i: (-frac[i], i))
    for i in order[:left]:
        out[i] += 1
    return out
