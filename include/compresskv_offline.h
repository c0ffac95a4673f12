/*
 * compresskv_offline.h -- C ABI of the offline analyses of CompressKV in
 * libcompresskv.so: the calibration that picks each layer's Semantic
 * Retrieval Heads (section 3.2, equation 1; section 3.3) and the estimate of
 * each layer's eviction error that sets the layer budgets (section 3.4,
 * equations 2-4).  Their outputs are the SRH masks and the budget vector that
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

#ifdef __cplusplus
}
#endif

#endif /* COMPRESSKV_OFFLINE_H */
