/*
 * compresskv.h -- C ABI of the MI355X (gfx950) CompressKV prefill-time KV-cache
 * eviction library (libcompresskv.so).
 *
 * The operation (CompressKV, section 3.3, with the SnapKV observation-window
 * setting of section 4): for every sequence b and KV group g of one layer,
 *   S1  logits of the last W queries of each Semantic Retrieval Head (SRH) of
 *       the group against every key of the sequence, causal inside the window;
 *   S2  softmax of every window row over its whole visible length;
 *   S3  sum of each SRH's attention over the W window rows, prefix keys only;
 *   S4  1-D pooling of that vector along the token axis, then the mean over
 *       the group's SRHs;
 *   S5  the (budget - W) best prefix tokens (ties: lowest position) plus the W
 *       window tokens, in ascending position order;
 *   S6  the retained K/V rows copied into a compact cache.
 * Budgets per layer come from an offline allocation (section 3.4) and the SRH
 * sets from an offline calibration (section 3.2, equation 1); both are inputs.
 *
 * Conventions shared by every entry point:
 *   - Pointers are DEVICE pointers unless the name ends in _host (host memory;
 *     a _ptrs_host array holds device pointers).  The caller
 *     owns every buffer; the library never allocates, frees or synchronizes.
 *   - All work is enqueued on `stream` (a hipStream_t; NULL = default stream).
 *     CKV_OK means "enqueued"; kernel faults surface at the caller's next sync.
 *     Buffers must stay alive until the stream has passed them.
 *   - Every argument is validated on the host before any HIP call; a failed
 *     check returns a nonzero status and enqueues nothing.  No exception
 *     crosses the ABI and nothing aborts.  compresskv_last_error() gives a
 *     thread-local description of the last failure.
 *   - Results are deterministic: the same inputs give the same bits.
 *   - Tensor layouts (elements, D = head_dim contiguous):
 *       q_win  [batch, W, n_q_heads, D]            dense
 *       k, v   [T, n_kv_heads, D] packed over the sequences of cu_seqlens,
 *              element (t, g, d) at t*stride_tok + g*stride_head + d
 *       scores [n_kv_heads, T] fp32                dense
 *       idx    [batch, n_kv_heads, budget] int32   dense
 *       k_out, v_out [batch, n_kv_heads, budget, D] dense, dtype of k / v
 *   - Query head h belongs to KV group h / (n_q_heads / n_kv_heads).
 */
#ifndef COMPRESSKV_H
#define COMPRESSKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* status codes */
#define CKV_OK 0
#define CKV_INVALID_ARGUMENT 1    /* null pointer, inconsistent sizes, budget < W, ... */
#define CKV_UNSUPPORTED 2         /* head_dim, dtype, alignment or size outside what the kernels take */
#define CKV_WORKSPACE_TOO_SMALL 3 /* ws_bytes < compresskv_workspace_bytes(...) */
#define CKV_HIP_ERROR 4           /* a kernel launch was rejected by the HIP runtime */

/* element types of q_win, k and v (all three share one) */
#define CKV_F32 0
#define CKV_BF16 1

/* pooling of the window sums along the token axis */
#define CKV_POOL_MAX 0 /* maximum over the in-range part of the window */
#define CKV_POOL_AVG 1 /* zero padding, divided by the kernel size */

/* order of pooling and SRH averaging */
#define CKV_POOL_THEN_MEAN 0 /* pool each SRH, then average (section 3.3) */
#define CKV_MEAN_THEN_POOL 1 /* average the SRH window sums, then pool once */

/* which heads share an index set */
#define CKV_INDEX_PER_GROUP 0 /* every KV group selects with its own SRHs (each group needs one) */
#define CKV_INDEX_LAYER 1     /* section 3.3: one selection per sequence from all the layer's SRHs
                                 (each against its own group's keys), kept by every group;
                                 groups without an SRH are allowed; CKV_POOL_THEN_MEAN only */

/* how S1-S4 are computed (the results agree within the scores' tolerance;
   each choice is deterministic) */
#define CKV_SCORE_AUTO 0     /* the library's choice (see compresskv_scoring_path) */
#define CKV_SCORE_TWO_PASS 1 /* two passes over K: row statistics, then window sums; in one
                                launch where the shape allows (see compresskv_scoring_path) */
#define CKV_SCORE_ONE_PASS 2 /* K read once; CKV_UNSUPPORTED where it does not apply */
#define CKV_SCORE_TWO_LAUNCHES 3 /* the two passes always in two launches (same bits as
                                    CKV_SCORE_TWO_PASS) */
#define CKV_SPIN_CATCHUP_ALL (-2) /* ckv_problem.spin_limit: see there */

/* Sizes and options of one layer.  head_dim must be 64 or 128. */
typedef struct ckv_problem {
  int32_t batch;        /* number of packed sequences, >= 1 */
  int32_t n_q_heads;    /* query heads Hq, a multiple of n_kv_heads, <= 256 */
  int32_t n_kv_heads;   /* KV groups Hkv, <= 128 */
  int32_t head_dim;     /* D: 64 or 128 */
  int32_t window;       /* W: observation-window length, >= 1 */
  int32_t dtype;        /* CKV_F32 or CKV_BF16 */
  int32_t pool_type;    /* CKV_POOL_MAX or CKV_POOL_AVG */
  int32_t pool_kernel;  /* odd, 1 .. 31 */
  int32_t reduce_order; /* CKV_POOL_THEN_MEAN or CKV_MEAN_THEN_POOL */
  float scale;          /* softmax scale; <= 0 selects 1/sqrt(head_dim) */
  const int32_t *cu_seqlens;      /* device [batch+1], cu[0] = 0, non-decreasing */
  const int32_t *cu_seqlens_host; /* host copy of the same offsets */
  int64_t k_stride_tok, k_stride_head; /* elements; each >= D (CKV_INVALID_ARGUMENT otherwise),
                                          multiples of 16 bytes (CKV_UNSUPPORTED otherwise) */
  int64_t v_stride_tok, v_stride_head;
  int32_t index_mode;   /* CKV_INDEX_PER_GROUP (0) or CKV_INDEX_LAYER */
  int32_t scoring;      /* CKV_SCORE_AUTO (0), _TWO_PASS, _ONE_PASS or _TWO_LAUNCHES */
  int32_t spin_limit;   /* single pass: how many times a unit polls for its segment's row
                           normalisers before it is left to the catch-up kernel that
                           follows on the same stream (about 1 us per poll); two passes in
                           one launch: how many times a workgroup polls for its group's
                           statistics before its column sums are left to the catch-up
                           kernel.  -1 (or any other negative value) selects the default
                           (64 single pass, 256 one launch), 0 never waits,
                           CKV_SPIN_CATCHUP_ALL leaves all of that work to the catch-up
                           kernel (to exercise that path).  Results do not depend on it. */
  int32_t reserved;     /* must be 0 */
} ckv_problem;

/*
 * Bytes of device workspace that compresskv_score / _select / _compress_layer
 * need for this problem, SRH mask (uint8 [n_q_heads], host) and budget.
 * Returns 0 if the arguments are invalid (see compresskv_last_error()).
 */
size_t compresskv_workspace_bytes(const ckv_problem *p, const uint8_t *srh_mask_host,
                                  int32_t budget);

/*
 * S1-S4: pooled, SRH-averaged score of every prefix token, per KV group.
 *   scores[g, t] for t in sequence b: the score of position t - cu[b] if that
 *   position is a prefix position (< L_b - W), +inf on the W window positions.
 *   With CKV_INDEX_LAYER every row g holds the layer score (the mean over all
 *   the layer's SRHs of their pooled window sums).
 * srh_mask_host: uint8 [n_q_heads]; every KV group needs at least one SRH
 *   (CKV_INDEX_LAYER: the layer needs one) and at most 16 row tiles
 *   (ceil(W/16) * n_srh <= 16; 12 for CKV_F32 at head_dim 128), else
 *   CKV_UNSUPPORTED.
 * Every sequence needs L_b >= W.  ws: >= compresskv_workspace_bytes(), any
 * contents, 256-byte aligned.
 */
int compresskv_score(const ckv_problem *p, const void *q_win, const void *k,
                     const uint8_t *srh_mask_host, float *scores, void *ws, size_t ws_bytes,
                     void *stream);

/*
 * S5: retained positions per (sequence, KV group), ascending, from scores laid
 * out as compresskv_score writes them (with CKV_INDEX_LAYER: one selection per
 * sequence from row 0, written into every group's row of idx).  If L_b <= budget all L_b positions
 * are kept; otherwise the (budget - W) highest prefix scores (ties: lowest
 * position) and the W window positions.  Entries past the kept count are -1.
 * Requires budget >= W.  Scores must be non-negative or +inf (NaN: undefined).
 */
int compresskv_select(const ckv_problem *p, const float *scores, int32_t budget, int32_t *idx,
                      void *ws, size_t ws_bytes, void *stream);

/*
 * S6: k_out[b, g, r, :] = k[cu[b] + idx[b, g, r], g, :] (same for v), bit for
 * bit; rows whose idx is -1 are written as zeros.  idx entries must be -1 or
 * in [0, L_b).
 */
int compresskv_gather(const ckv_problem *p, const void *k, const void *v, const int32_t *idx,
                      int32_t budget, void *k_out, void *v_out, void *stream);

/*
 * S1-S6 for one layer: score, select and gather in one call.  scores_or_null
 * receives the scores when not NULL (otherwise they live in ws).
 */
int compresskv_compress_layer(const ckv_problem *p, const void *q_win, const void *k,
                              const void *v, const uint8_t *srh_mask_host, int32_t budget,
                              int32_t *idx, void *k_out, void *v_out, float *scores_or_null,
                              void *ws, size_t ws_bytes, void *stream);

/*
 * compresskv_compress_layer without a workspace argument and without any
 * allocation, for callers that can not allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc).
 * The library's scratch is a fixed array of 32 MiB per device, held from the
 * first call on that device until the process ends; a problem whose
 * compresskv_workspace_bytes exceeds it returns CKV_WORKSPACE_TOO_SMALL (use
 * compresskv_compress_layer with a workspace).  Every call on one device
 * shares that device's array: calls that overlap in time on one device (other
 * streams, other threads) race and must be serialised by the caller.  Results
 * are identical to compresskv_compress_layer's.  The first call on a device
 * looks up the array's address (hipGetSymbolAddress) with that device current.
 */
int compresskv_compress_layer_noalloc(const ckv_problem *p, const void *q_win, const void *k,
                                      const void *v, const uint8_t *srh_mask_host,
                                      int32_t budget, int32_t *idx, void *k_out, void *v_out,
                                      float *scores_or_null, void *stream);

/*
 * Multi-layer calls.  A model's layers share one problem (shapes, cu_seqlens,
 * strides, options) and differ in their operands, SRH masks and budgets
 * (section 3.4 gives every layer its own budget; section 3.2 every layer its
 * own SRHs).  Per-layer DEVICE pointers are passed in HOST arrays of n_layers
 * entries (names ending in _ptrs_host); srh_masks_host is uint8
 * [n_layers][n_q_heads] and budgets_host int32 [n_layers], both host memory.
 * Every layer is validated before anything is enqueued; the work of all
 * layers is enqueued as a few launches (each kernel covers every layer), so
 * per-layer launch costs and the HBM ramp of a kernel are paid once per call.
 * Results are bit-identical to per-layer compresskv_compress_layer calls.
 * n_layers * batch <= 65535.
 */

/* Workspace bytes of the multi-layer calls for this problem and these masks
 * (independent of the budgets).  0 on invalid arguments. */
size_t compresskv_layers_workspace_bytes(const ckv_problem *p, int32_t n_layers,
                                         const uint8_t *srh_masks_host);

/*
 * S1-S4 for n_layers layers: scores [n_layers][n_kv_heads][T] fp32 (device),
 * layer l laid out as compresskv_score writes it.  Each layer's SRH groups
 * obey compresskv_score's limit (ceil(W/16) * SRHs per group <= 16, or 12).
 */
int compresskv_score_layers(const ckv_problem *p, int32_t n_layers,
                            const void *const *q_win_ptrs_host, const void *const *k_ptrs_host,
                            const uint8_t *srh_masks_host, float *scores, void *ws,
                            size_t ws_bytes, void *stream);

/*
 * S1-S6 for n_layers layers (the per-layer budget vector of the method): layer
 * l reads q_win_ptrs_host[l], k_ptrs_host[l], v_ptrs_host[l] and writes
 * idx_ptrs_host[l] [batch, n_kv_heads, budgets_host[l]] and k_out/v_out
 * [batch, n_kv_heads, budgets_host[l], D] as compresskv_compress_layer does.
 * scores_or_null: NULL or device [n_layers][n_kv_heads][T] fp32.
 */
int compresskv_compress_layers(const ckv_problem *p, int32_t n_layers,
                               const void *const *q_win_ptrs_host, const void *const *k_ptrs_host,
                               const void *const *v_ptrs_host, const uint8_t *srh_masks_host,
                               const int32_t *budgets_host, int32_t *const *idx_ptrs_host,
                               void *const *k_out_ptrs_host, void *const *v_out_ptrs_host,
                               float *scores_or_null, void *ws, size_t ws_bytes, void *stream);

/*
 * Head-level budgets (per-group budgets, as in the combination of CompressKV
 * with head-level allocation, section 4 "Orthogonal to Prior Efficiency
 * Methods"): KV group g keeps group_budgets_host[g] (>= W) positions, chosen
 * exactly as by compresskv_select with that budget.  The outputs are ragged
 * per group: with off[g] = the sum of the budgets of groups 0 .. g-1 and
 * total = the sum of all of them,
 *   idx    int32 [batch][total]:   entry j of (b, g) at b * total + off[g] + j
 *   k_out, v_out [batch][total][D]: row b * total + off[g] + j, dtype of k / v
 * with -1 / zero rows past a group's kept count.  Needs CKV_INDEX_PER_GROUP
 * (CKV_UNSUPPORTED otherwise) and batch * total < 2^31.  The workspace of
 * compresskv_compress_layer_heads is compresskv_workspace_bytes(p, mask,
 * max_g group_budgets_host[g]).
 */
int compresskv_select_heads(const ckv_problem *p, const float *scores,
                            const int32_t *group_budgets_host, int32_t *idx, void *stream);
int compresskv_gather_heads(const ckv_problem *p, const void *k, const void *v,
                            const int32_t *idx, const int32_t *group_budgets_host, void *k_out,
                            void *v_out, void *stream);
int compresskv_compress_layer_heads(const ckv_problem *p, const void *q_win, const void *k,
                                    const void *v, const uint8_t *srh_mask_host,
                                    const int32_t *group_budgets_host, int32_t *idx, void *k_out,
                                    void *v_out, float *scores_or_null, void *ws, size_t ws_bytes,
                                    void *stream);

/*
 * Which scoring implementation compresskv_score / _compress_layer will use for
 * this problem: 1 = single pass (each key read once from HBM), 2 = two passes
 * over K in two launches (statistics, then column sums), 3 = the same two
 * passes in one launch (each group's column-sum workgroups wait inside the
 * launch for its statistics; same bits as 2).  CKV_SCORE_TWO_PASS uses one
 * launch for bf16 inputs with at most 8 row tiles per group, else two;
 * CKV_SCORE_AUTO uses one launch for bf16 inputs with at most 6 row tiles
 * per group where every sequence also spans at least 16 statistics chunks
 * (about 8k-16k keys; shorter sequences leave most of the one launch's
 * workgroups idle), else two launches (the faster on the measured shapes;
 * the single pass is slower than either);
 * CKV_SCORE_TWO_LAUNCHES always uses two launches; CKV_SCORE_ONE_PASS uses
 * the single pass, which needs bf16 inputs, CKV_INDEX_PER_GROUP, batch <= 64
 * and at most 6 row tiles per group (ceil(W/16) * SRHs), and otherwise
 * returns -CKV_UNSUPPORTED.  The multi-layer calls make the same choice over
 * all their layers (single pass: layer by layer).  Negative on invalid
 * arguments (minus the status).
 */
int compresskv_scoring_path(const ckv_problem *p, const uint8_t *srh_mask_host);

/* Static text of a status code. */
const char *compresskv_status_string(int status);

/* Thread-local description of the last failure of this thread ("" if none). */
const char *compresskv_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* COMPRESSKV_H */
