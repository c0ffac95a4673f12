"""Plain, slow, fp64 CPU oracle for CompressKV's prefill-time KV-cache eviction.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import or call this module.  The
product path (the HIP library and its Python binding) never touches it, and
this module imports nothing from the product package.

What it computes (CompressKV, section 3.3 "Token selection driven by Semantic
Retrieval Heads", with the SnapKV local-window setting of section 4,
"Implementation Details"):

  for every sequence b and every KV group g of one layer (per-group mode; the
  layer-shared mode averages the pooled vectors of all the layer's SRHs and
  keeps one index set for every group)
    1. attention of the last W prompt queries of each Semantic Retrieval Head
       (SRH) h of the group against all keys of the prompt, causal inside the
       window, softmax over the whole row;
    2. sum of that attention over the W window queries (prefix keys only);
    3. 1-D pooling of that vector along the token axis (stride 1, odd kernel);
    4. mean of the pooled vectors over the group's SRHs;
    5. the (budget - W) highest-scoring prefix tokens (ties: lowest index),
       plus the W window tokens, in ascending position order;
    6. the retained K/V rows copied into a compact cache.

Every step is written straight from its definition in float64 with numpy; no
blocking, fusion or reordering.  Readings of points the paper leaves open are
listed in the repository's design notes and restated where they are used:

  * per-group selection (one index set per KV group, from that group's SRHs);
  * the budget counts the W window tokens;
  * softmax scale 1/sqrt(D) unless given, applied to the exact dot product;
  * max pooling ignores out-of-range positions, average pooling pads with
    zeros and divides by the kernel size (count_include_pad);
  * pooling never reads window positions; window positions score +inf;
  * ties are broken by the lowest position;
  * query head h belongs to KV group h // (Hq // Hkv).

Parity status: every function here is pinned by the CPU tests
(brute-force attention, exact rational worked examples, library routines,
closed forms, invariants and metamorphic relations).  The paper prints no
numeric worked example of this path, so agreement with the paper's own
numbers is unpinned; the pins are mathematical.
"""
from __future__ import annotations

import math
from dataclasses import dataclass

import numpy as np

POOL_MAX = 0
POOL_AVG = 1
POOL_THEN_MEAN = 0
MEAN_THEN_POOL = 1
PER_GROUP = 0       # one index set per KV group, chosen by that group's SRHs
LAYER_SHARED = 1    # one index set for every head of the layer (section 3.3)


# --------------------------------------------------------------------------
# Step 1: observation-window attention of one head (section 3.3: the SRH
# attention matrices follow SnapKV, i.e. the attention of the last window
# queries over the prompt).
# --------------------------------------------------------------------------
def window_logits(q_head: np.ndarray, k_seq: np.ndarray, scale: float) -> np.ndarray:
    """Scaled logits of the W window queries of one head against all L keys.

    q_head: [W, D] float64, the last W queries (positions L-W .. L-1).
    k_seq:  [L, D] float64, every key of the sequence for this head's group.
    Returns Z [W, L]; Z[i, j] = -inf where key j lies after query i
    (j > P + i with P = L - W), i.e. causal attention.
    """
    W = q_head.shape[0]
    L = k_seq.shape[0]
    P = L - W
    z = scale * (q_head @ k_seq.T)
    for i in range(W):
        z[i, P + i + 1:] = -np.inf
    return z


def row_softmax(z: np.ndarray) -> np.ndarray:
    """Softmax of every row over all its unmasked entries (window keys included)."""
    m = np.max(z, axis=1, keepdims=True)
    e = np.exp(z - m)
    return e / np.sum(e, axis=1, keepdims=True)


# --------------------------------------------------------------------------
# Step 2: sum over the observation window (section 3.3: each SRH attention
# matrix is reduced by adding up its window rows).  Only prefix keys are
# scored: window keys are always kept and never ranked.
# --------------------------------------------------------------------------
def window_column_sums(a: np.ndarray, P: int) -> np.ndarray:
    """c[j] = sum_i A[i, j] for the prefix keys j < P."""
    return np.sum(a[:, :P], axis=0)


# --------------------------------------------------------------------------
# Step 3: 1-D pooling along the token axis (section 3.3, the SnapKV-style
# clustering step; kernel size 5 in the paper's setting, section 4).
# --------------------------------------------------------------------------
def pool1d(c: np.ndarray, kernel: int, kind: int) -> np.ndarray:
    """Stride-1 'same' pooling of a length-P vector with an odd kernel.

    max: maximum over the in-range part of [j - r, j + r];
    avg: sum over the in-range part divided by the kernel size.
    """
    if kernel < 1 or kernel % 2 == 0:
        raise ValueError("pool kernel must be odd and >= 1")
    P = c.shape[0]
    r = (kernel - 1) // 2
    out = np.empty(P, dtype=np.float64)
    for j in range(P):
        lo = max(0, j - r)
        hi = min(P, j + r + 1)
        if kind == POOL_MAX:
            out[j] = np.max(c[lo:hi])
        elif kind == POOL_AVG:
            out[j] = np.sum(c[lo:hi]) / kernel
        else:
            raise ValueError("unknown pool kind")
    return out


# --------------------------------------------------------------------------
# Steps 1-4 for one KV group: per-SRH scores, pooled, then averaged over the
# group's SRHs (section 3.3: the pooled vectors of the SRHs are averaged).
# --------------------------------------------------------------------------
def group_scores(q_heads: list[np.ndarray], k_seq: np.ndarray, scale: float,
                 pool_kernel: int, pool_type: int = POOL_MAX,
                 reduce_order: int = POOL_THEN_MEAN) -> np.ndarray:
    """Score of every prefix token of one sequence for one KV group.

    q_heads: list of [W, D] window queries, one per SRH of the group.
    k_seq:   [L, D] keys of the group.
    reduce_order POOL_THEN_MEAN pools each head and then averages (the
    paper's order); MEAN_THEN_POOL averages the window sums first.
    """
    W = q_heads[0].shape[0]
    L = k_seq.shape[0]
    P = L - W
    sums = []
    for q in q_heads:
        a = row_softmax(window_logits(q, k_seq, scale))
        sums.append(window_column_sums(a, P))
    if reduce_order == POOL_THEN_MEAN:
        pooled = [pool1d(c, pool_kernel, pool_type) for c in sums]
        return np.mean(np.stack(pooled), axis=0) if P > 0 else np.zeros(0)
    if reduce_order == MEAN_THEN_POOL:
        if P == 0:
            return np.zeros(0)
        return pool1d(np.mean(np.stack(sums), axis=0), pool_kernel, pool_type)
    raise ValueError("unknown reduce order")


# --------------------------------------------------------------------------
# Steps 1-4 for a whole layer with one shared index set (section 3.3: the
# layer's top SRHs, each attending to its own group's keys, are compressed by
# the window sum and pooling, and the compressed vectors are averaged; every
# head of the layer then keeps the same tokens).  Pool each SRH, then average
# (the paper's order).
# --------------------------------------------------------------------------
def layer_scores(q_and_keys: list[tuple[np.ndarray, np.ndarray]], scale: float,
                 pool_kernel: int, pool_type: int = POOL_MAX) -> np.ndarray:
    """Score of every prefix token of one sequence for the whole layer.

    q_and_keys: one (q [W, D], k [L, D]) pair per SRH of the layer, k being
    the keys of the SRH's own KV group.
    """
    W = q_and_keys[0][0].shape[0]
    L = q_and_keys[0][1].shape[0]
    P = L - W
    if P == 0:
        return np.zeros(0)
    pooled = []
    for q, k_seq in q_and_keys:
        a = row_softmax(window_logits(q, k_seq, scale))
        pooled.append(pool1d(window_column_sums(a, P), pool_kernel, pool_type))
    return np.mean(np.stack(pooled), axis=0)


# --------------------------------------------------------------------------
# Step 5: budgeted top-N that always keeps the window (section 3.3: the N
# best-scoring tokens keep their KV pairs, the rest are evicted; the window
# is kept as in SnapKV, section 4).
# --------------------------------------------------------------------------
def select_tokens(score: np.ndarray, L: int, window: int, budget: int) -> np.ndarray:
    """Retained positions of one sequence/group, ascending.

    The budget counts the window.  If L <= budget every token is kept.
    Otherwise the (budget - window) best prefix tokens are kept, ranked by
    score descending and position ascending, followed by the window.
    """
    if budget < window or L < window:
        raise ValueError("budget and sequence length must be at least the window")
    if L <= budget:
        return np.arange(L, dtype=np.int64)
    P = L - window
    n_top = budget - window
    order = np.lexsort((np.arange(P), -score))
    top = np.sort(order[:n_top])
    return np.concatenate([top, np.arange(P, L)]).astype(np.int64)


# --------------------------------------------------------------------------
# Whole layer.
# --------------------------------------------------------------------------
@dataclass
class LayerResult:
    idx: np.ndarray      # [batch, Hkv, budget] int64; -1 past the kept count
    k_out: np.ndarray    # [batch, Hkv, budget, D], same dtype as k; zeros past the kept count
    v_out: np.ndarray
    scores: np.ndarray   # [Hkv, T] float64; +inf on window positions


def compress_layer(q_win: np.ndarray, k: np.ndarray, v: np.ndarray,
                   cu_seqlens: np.ndarray, srh_mask: np.ndarray, budget: int,
                   pool_kernel: int, pool_type: int = POOL_MAX,
                   reduce_order: int = POOL_THEN_MEAN, scale: float | None = None,
                   k_values: np.ndarray | None = None,
                   q_values: np.ndarray | None = None,
                   index_mode: int = PER_GROUP) -> LayerResult:
    """CompressKV eviction of one layer.

    q_win: [batch, W, Hq, D] window queries (any float dtype, or raw bits when
           q_values gives the float64 values).
    k, v:  [T, Hkv, D] packed keys/values of all sequences (any dtype; copied
           bit for bit).  k_values, if given, are k's values as float64
           (needed when k holds raw bf16 bits).
    cu_seqlens: [batch+1] offsets of the sequences in the packed T axis.
    srh_mask: [Hq] nonzero for Semantic Retrieval Heads.
    index_mode: PER_GROUP (each KV group selects with its own SRHs; every
        group needs one) or LAYER_SHARED (one selection from all the layer's
        SRHs, kept by every group; pool-then-mean only; scores[g] then holds
        the layer score for every g).
    """
    qv = np.asarray(q_values if q_values is not None else q_win, dtype=np.float64)
    kv = np.asarray(k_values if k_values is not None else k, dtype=np.float64)
    batch, W, Hq, D = qv.shape
    T, Hkv, _ = kv.shape
    G = Hq // Hkv
    if scale is None or scale <= 0:
        scale = 1.0 / math.sqrt(D)
    idx = np.full((batch, Hkv, budget), -1, dtype=np.int64)
    k_out = np.zeros((batch, Hkv, budget, D), dtype=k.dtype)
    v_out = np.zeros((batch, Hkv, budget, D), dtype=v.dtype)
    scores = np.zeros((Hkv, T), dtype=np.float64)
    if index_mode == LAYER_SHARED:
        if reduce_order != POOL_THEN_MEAN:
            raise ValueError("the layer-shared index set pools each SRH, then averages")
        srh = [h for h in range(Hq) if srh_mask[h]]
        if not srh:
            raise ValueError("the layer has no Semantic Retrieval Head")
        for b in range(batch):
            s0, s1 = int(cu_seqlens[b]), int(cu_seqlens[b + 1])
            L = s1 - s0
            P = L - W
            sc = layer_scores([(qv[b, :, h, :], kv[s0:s1, h // G, :]) for h in srh], scale,
                              pool_kernel, pool_type)
            sel = select_tokens(sc, L, W, budget)
            n = sel.shape[0]
            for g in range(Hkv):
                scores[g, s0:s0 + P] = sc
                scores[g, s0 + P:s1] = np.inf
                idx[b, g, :n] = sel
                k_out[b, g, :n] = k[s0 + sel, g, :]
                v_out[b, g, :n] = v[s0 + sel, g, :]
        return LayerResult(idx=idx, k_out=k_out, v_out=v_out, scores=scores)
    if index_mode != PER_GROUP:
        raise ValueError("unknown index mode")
    for b in range(batch):
        s0, s1 = int(cu_seqlens[b]), int(cu_seqlens[b + 1])
        L = s1 - s0
        P = L - W
        for g in range(Hkv):
            heads = [h for h in range(g * G, (g + 1) * G) if srh_mask[h]]
            if not heads:
                raise ValueError(f"KV group {g} has no Semantic Retrieval Head")
            q_heads = [qv[b, :, h, :] for h in heads]
            sc = group_scores(q_heads, kv[s0:s1, g, :], scale, pool_kernel,
                              pool_type, reduce_order)
            scores[g, s0:s0 + P] = sc
            scores[g, s0 + P:s1] = np.inf
            sel = select_tokens(sc, L, W, budget)
            n = sel.shape[0]
            idx[b, g, :n] = sel
            k_out[b, g, :n] = k[s0 + sel, g, :]
            v_out[b, g, :n] = v[s0 + sel, g, :]
    return LayerResult(idx=idx, k_out=k_out, v_out=v_out, scores=scores)


def compress_layer_heads(q_win: np.ndarray, k: np.ndarray, v: np.ndarray,
                         cu_seqlens: np.ndarray, srh_mask: np.ndarray,
                         group_budgets: np.ndarray, pool_kernel: int,
                         pool_type: int = POOL_MAX, reduce_order: int = POOL_THEN_MEAN,
                         scale: float | None = None,
                         k_values: np.ndarray | None = None) -> LayerResult:
    """Per-group budgets (head-level budget allocation, combined with CompressKV
    in section 4 "Orthogonal to Prior Efficiency Methods"): group g keeps
    group_budgets[g] tokens, chosen exactly as in compress_layer.

    The outputs are ragged per group: with off[g] = sum of the budgets of the
    groups before g, idx[b, off[g] + j] is group g's j-th kept position and
    k_out[b, off[g] + j] its row (-1 / zeros past the kept count).
    scores are those of compress_layer (they do not depend on the budget).
    """
    group_budgets = np.asarray(group_budgets, dtype=np.int64)
    Hkv = k.shape[1]
    batch, D = q_win.shape[0], k.shape[2]
    off = np.concatenate([[0], np.cumsum(group_budgets)])
    total = int(off[-1])
    idx = np.full((batch, total), -1, dtype=np.int64)
    k_out = np.zeros((batch, total, D), dtype=k.dtype)
    v_out = np.zeros((batch, total, D), dtype=v.dtype)
    scores = None
    for g in range(Hkv):
        res = compress_layer(q_win, k, v, cu_seqlens, srh_mask, int(group_budgets[g]),
                             pool_kernel, pool_type, reduce_order, scale=scale,
                             k_values=k_values)
        if scores is None:
            scores = res.scores
        o = int(off[g])
        idx[:, o:o + int(group_budgets[g])] = res.idx[:, g]
        k_out[:, o:o + int(group_budgets[g])] = res.k_out[:, g]
        v_out[:, o:o + int(group_budgets[g])] = res.v_out[:, g]
    return LayerResult(idx=idx, k_out=k_out, v_out=v_out, scores=scores)

