/*
 * compresskv_offline.h -- C ABI of the offline analyses of CompressKV in
 * libcompresskv.so: the calibration that picks each layer's Semantic
 * Retrieval Heads (section 3.2, equation 1; section 3.3), the estimate of
 * each layer's eviction error (section 3.4, equations 2-4) and the layer
 * budgets set from it (section 3.4, limits of section 4).  Their outputs are the SRH masks and the budget vector that
 * the eviction entry points of compresskv.h take.
 *
 * The conventions of compresskv.h hold here too: device pointers unless the
 * name ends in _host, caller-owned memory, work enqueued on `stream`,
 * validation on the host before any HIP call, status codes CKV_*,
 * compresskv_last_error() for the reason of a failure, deterministic results.
 */
#ifndef COMPRESSKV_OFFLINE_H
#define COMPRESSKV_OFFLINE_H

#include "compresskv.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Sizes of an SRH calibration run. */
typedef struct ckv_srh_problem {
  int32_t n_samples;          /* S >= 1 calibration samples */
  int32_t n_steps;            /* N >= 1 decoding steps per sample */
  int32_t n_heads;            /* H >= 1 attention heads, all layers, layer-major */
  int32_t ctx_len;            /* L >= 1 context positions per sample */
  const int32_t *spans_host;  /* [S][2] answer span (start, length) of each sample:
                                 start >= 0, length >= 1, start + length <= L */
} ckv_srh_problem;

/*
 * Equation 1 (section 3.2): the SRH score of every head,
 *   scores[h] = sum over samples s and steps t whose generated token
 *               gen_tokens[s][t] equals the token id at some position of the
 *               answer span (ctx_tokens[s][start .. start+length)) of
 *               sum over the span positions j of attn[s][t][h][j].
 * attn       fp32 [S][N][H][L] dense: head h's attention weights at step t.
 * gen_tokens int32 [S][N]; ctx_tokens int32 [S][L]; spans int32 [S][2] (the
 *            device copy of spans_host).
 * scores     fp32 [H] (written).  Each head's sum runs in a fixed order: per
 *            step in fp32, over steps and samples in fp64.
 */
int compresskv_srh_scores(const ckv_srh_problem *p, const float *attn, const int32_t *gen_tokens,
                          const int32_t *ctx_tokens, const int32_t *spans, float *scores,
                          void *stream);

/*
 * Section 3.3: every layer's SRH set, its top_k heads by score (ties: lower
 * head index).  scores fp32 [n_layers][heads_per_layer] (as written by
 * compresskv_srh_scores, layer-major); srh_mask uint8 [n_layers][heads_per_layer]
 * (written: 1 for an SRH).  Requires 1 <= top_k <= heads_per_layer <= 1024.
 * Scores must not be NaN (NaN: undefined ranking).
 */
int compresskv_select_srh(int32_t n_layers, int32_t heads_per_layer, const float *scores,
                          int32_t top_k, uint8_t *srh_mask, void *stream);

/* Sizes of one layer's eviction-error estimate (the layer's shapes, dtype,
   strides, cu_seqlens and softmax scale come from its ckv_problem). */
typedef struct ckv_error_problem {
  int32_t n_steps;   /* T >= 1 decoding steps per sequence (the kernels take blocks of
                        steps and sequences; T is bounded by the workspace only) */
  int32_t d_model;   /* rows of W_O, >= 1 */
  int32_t budget;    /* B: rows per (sequence, group) of k_out / v_out, >= 1 */
  float eps;         /* >= 0, e.g. 1e-6 */
} ckv_error_problem;

size_t compresskv_layer_error_workspace_bytes(const ckv_problem *p, const ckv_error_problem *e);

/*
 * Equations 2-4 (section 3.4): the eviction error of one layer,
 *   err[0] = sum over sequences b and steps t of
 *            ||W_O (A_full - A_comp)||_F / (||W_O A_full||_F + eps)
 * where A_full[b][t] is the softmax attention of the step's queries (every
 * query head, head h over KV group h / (n_q_heads / n_kv_heads)) over the full
 * cache k, v of sequence b, A_comp the same over the compact cache, and the
 * heads' outputs are concatenated head-major (h * head_dim + d).
 * q_dec  [batch][T][n_q_heads][head_dim], dtype of the problem.
 * k, v   the full caches, laid out as for compresskv_compress_layer.
 * k_out, v_out  [batch][n_kv_heads][budget][head_dim]: the compact caches as
 *        compresskv_compress_layer writes them; the first min(L_b, budget) rows
 *        of each (sequence, group) are the kept positions.
 * w_o    [d_model][n_q_heads * head_dim], dtype of the problem;
 *        n_q_heads * head_dim must be a multiple of 256.
 * err    fp32 [1] (written).  The decoding steps' own tokens are in neither
 *        cache, so the two attentions differ only by the eviction.
 * ws:    >= compresskv_layer_error_workspace_bytes(), 256-byte aligned.
 */
int compresskv_layer_error(const ckv_problem *p, const ckv_error_problem *e, const void *q_dec,
                           const void *k, const void *v, const void *k_out, const void *v_out,
                           const void *w_o, float *err, void *ws, size_t ws_bytes, void *stream);

/*
 * Section 3.4 with the limits of section 4: integer layer budgets from the
 * layers' errors.  Every layer gets min_budget; the rest of `total` goes to
 * the layers in proportion to their normalised errors (errors / sum);
 * layers that would pass max_budget are held there and their excess is
 * shared again among the others; units left over by rounding down go one each
 * to the largest fractional shares (ties: lower layer).  Host memory only
 * (no GPU work): errors_host float [n_layers] (>= 0, finite, not all 0
 * unless every layer gets an even share), budgets_host int32 [n_layers]
 * (written).  Requires n_layers * min_budget <= total <= n_layers * max_budget
 * and 1 <= min_budget <= max_budget.
 */
int compresskv_allocate_budgets(int32_t n_layers, const float *errors_host, int64_t total,
                                int32_t min_budget, int32_t max_budget, int32_t *budgets_host);

#ifdef __cplusplus
}
#endif

#endif /* COMPRESSKV_OFFLINE_H */
