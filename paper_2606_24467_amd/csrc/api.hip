// C ABI of libcompresskv: host-side validation, workspace layout and dispatch.
// Every check runs before the first HIP call, so invalid arguments never touch
// the device and can be tested without a GPU.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/compresskv.h"
#include "api_common.h"
#include "ckv_launch.h"

namespace {

using ckv_api::aligned;
using ckv_api::fail;
using ckv_api::g_last_error;
using ckv_api::ok;

int elem_size(const ckv_problem *p) { return p->dtype == CKV_BF16 ? 2 : 4; }

// SRH lists of one layer, from its host mask.
struct LayerSrh {
  std::vector<uint16_t> off;   // [Hkv + 1]
  std::vector<uint8_t> head;   // [n SRHs]
  int nmax = 0;                // most SRHs in one group
};

// Everything derived from a validated problem and its SRH masks.
struct Plan {
  int64_t T = 0;
  int lmax = 0;
  int n_layers = 1;    // layers of the call (1 for single-layer calls)
  int th = 0;          // row tiles per SRH
  int rt_max = 0;      // max row tiles of a group (over the layers)
  int nmax = 0;        // most SRHs in one group (over the layers)
  std::vector<int> rt_layer;   // max row tiles of a group, per layer
  int chunk1 = 0, max_chunks1 = 0;
  int chunk2 = 0, max_chunks2 = 0;
  int cpw1 = 1, cpw2 = 1;  // consecutive chunks per leading scoring workgroup
  int lead1 = 1, lead2 = 1;  // leading workgroups per (sequence, group) and layer
  uint32_t head_end_mask = 0;
  // workspace: table | scores | counters (ticket, arrivals, normalisers,
  // histograms) | partial statistics | skip list | edge window sums | the
  // one-launch form's catch-up list | split-selection slices
  size_t table_off = 0, scores_off = 0, counters_off = 0, arrive_off = 0, bias_off = 0,
         hist_off = 0, stats_off = 0, skip_off = 0, edges_off = 0, total = 0;
  int64_t stats_layer = 0, hist_layer = 0;   // elements per layer
  int sel_slices = 0;      // slices of the split selection (0: one workgroup per selection)
  size_t sel_meta_off = 0, sel_cand_off = 0, sel_ord_off = 0;
  int max_parts = 0;       // partial-statistics slots per group in the workspace
  // single-pass scoring
  bool op_shape = false;   // the problem's shape allows it (its workspace is reserved)
  int units_layer = 0;     // its units per layer
  int ew = 0;              // window sums kept at each end of a unit
  int n_op = 0;            // layers scored in a single pass: the first n_op table entries
  int op_rt_max = 0, tp_rt_max = 0;   // row tiles of those layers / of the others
  int op_grid = 0;         // persistent workgroups of the single-pass kernel
  // two-pass scoring in one launch (fused_kernel)
  bool fused = false;
  size_t fskip_off = 0;    // its catch-up list: count, then workgroup indices
  std::vector<int> order;  // table entry -> caller's layer (single-pass layers first)
  LayerSrh srh;            // single-layer calls
};

// Keys per workgroup: the smallest power of two >= lo such that doubling it
// would leave fewer than `target` workgroups for one layer, capped at hi.  It
// depends on the layer's shape only: the chunking fixes the merge order of the
// partial row statistics, so multi-layer calls reproduce single-layer bits.
int pick_chunk(const ckv_problem *p, int lo, int hi, int target) {
  int c = lo;
  while (c < hi) {
    int64_t wg = 0;
    for (int b = 0; b < p->batch; ++b) {
      const int L = p->cu_seqlens_host[b + 1] - p->cu_seqlens_host[b];
      wg += (L + 2 * c - 1) / (2 * c);
    }
    wg *= p->n_kv_heads;
    if (wg < target) break;
    c *= 2;
  }
  return c;
}

size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Shape and option checks shared by every entry point.
int check_problem(const ckv_problem *p) {
  if (!p) return fail(CKV_INVALID_ARGUMENT, "problem is NULL");
  if (p->batch < 1) return fail(CKV_INVALID_ARGUMENT, "batch must be >= 1 (got %d)", p->batch);
  if (p->n_kv_heads < 1 || p->n_q_heads < 1)
    return fail(CKV_INVALID_ARGUMENT, "head counts must be >= 1");
  if (p->n_q_heads % p->n_kv_heads != 0)
    return fail(CKV_INVALID_ARGUMENT, "n_q_heads (%d) must be a multiple of n_kv_heads (%d)",
                p->n_q_heads, p->n_kv_heads);
  if (p->n_kv_heads > ckv::kMaxKvHeads || p->n_q_heads > ckv::kMaxQHeads)
    return fail(CKV_UNSUPPORTED, "at most %d KV heads and %d query heads", ckv::kMaxKvHeads,
                ckv::kMaxQHeads);
  if (p->head_dim != 64 && p->head_dim != 128)
    return fail(CKV_UNSUPPORTED, "head_dim must be 64 or 128 (got %d)", p->head_dim);
  if (p->dtype != CKV_F32 && p->dtype != CKV_BF16)
    return fail(CKV_UNSUPPORTED, "dtype must be CKV_F32 or CKV_BF16 (got %d)", p->dtype);
  if (p->window < 1) return fail(CKV_INVALID_ARGUMENT, "window must be >= 1 (got %d)", p->window);
  if (p->pool_type != CKV_POOL_MAX && p->pool_type != CKV_POOL_AVG)
    return fail(CKV_INVALID_ARGUMENT, "pool_type must be CKV_POOL_MAX or CKV_POOL_AVG");
  if (p->pool_kernel < 1 || p->pool_kernel % 2 == 0 || p->pool_kernel > ckv::kMaxPoolKernel)
    return fail(CKV_INVALID_ARGUMENT, "pool_kernel must be odd and in [1, %d] (got %d)",
                ckv::kMaxPoolKernel, p->pool_kernel);
  if (p->reduce_order != CKV_POOL_THEN_MEAN && p->reduce_order != CKV_MEAN_THEN_POOL)
    return fail(CKV_INVALID_ARGUMENT, "reduce_order must be CKV_POOL_THEN_MEAN or CKV_MEAN_THEN_POOL");
  if (!(std::isfinite(p->scale)))
    return fail(CKV_INVALID_ARGUMENT, "scale must be finite");
  if (p->index_mode != CKV_INDEX_PER_GROUP && p->index_mode != CKV_INDEX_LAYER)
    return fail(CKV_INVALID_ARGUMENT, "index_mode must be CKV_INDEX_PER_GROUP or CKV_INDEX_LAYER");
  if (p->scoring != CKV_SCORE_AUTO && p->scoring != CKV_SCORE_TWO_PASS &&
      p->scoring != CKV_SCORE_ONE_PASS && p->scoring != CKV_SCORE_TWO_LAUNCHES)
    return fail(CKV_INVALID_ARGUMENT, "scoring must be CKV_SCORE_AUTO, CKV_SCORE_TWO_PASS, "
                                      "CKV_SCORE_ONE_PASS or CKV_SCORE_TWO_LAUNCHES");
  if (p->reserved != 0) return fail(CKV_INVALID_ARGUMENT, "reserved must be 0");
  if (p->index_mode == CKV_INDEX_LAYER && p->reduce_order != CKV_POOL_THEN_MEAN)
    return fail(CKV_UNSUPPORTED, "CKV_INDEX_LAYER needs reduce_order CKV_POOL_THEN_MEAN");
  if (!p->cu_seqlens || !p->cu_seqlens_host)
    return fail(CKV_INVALID_ARGUMENT, "cu_seqlens and cu_seqlens_host are both required");
  if (!aligned(p->cu_seqlens, 4)) return fail(CKV_UNSUPPORTED, "cu_seqlens must be 4-byte aligned");
  if (p->cu_seqlens_host[0] != 0) return fail(CKV_INVALID_ARGUMENT, "cu_seqlens[0] must be 0");
  for (int b = 0; b < p->batch; ++b) {
    const int L = p->cu_seqlens_host[b + 1] - p->cu_seqlens_host[b];
    if (L < 0) return fail(CKV_INVALID_ARGUMENT, "cu_seqlens is decreasing at %d", b);
    if (L < p->window)
      return fail(CKV_INVALID_ARGUMENT, "sequence %d has length %d < window %d", b, L, p->window);
  }
  const int es = elem_size(p);
  const int64_t strides[4] = {p->k_stride_tok, p->k_stride_head, p->v_stride_tok, p->v_stride_head};
  static const char *const names[4] = {"k_stride_tok", "k_stride_head", "v_stride_tok",
                                       "v_stride_head"};
  for (int i = 0; i < 4; ++i) {
    if (strides[i] < p->head_dim)
      return fail(CKV_INVALID_ARGUMENT, "%s (%lld) must be >= head_dim (%d)", names[i],
                  (long long)strides[i], p->head_dim);
    if ((strides[i] * es) % 16 != 0)
      return fail(CKV_UNSUPPORTED, "K/V strides must be multiples of 16 bytes");
  }
  return CKV_OK;
}

// Per-group SRH lists of one layer from its host mask (`layer` only names it
// in messages).  Every group needs an SRH, except with the layer-shared index
// set, which needs one in the layer.
int layer_srh(const ckv_problem *p, const uint8_t *mask, int layer, LayerSrh &ls) {
  if (!mask) return fail(CKV_INVALID_ARGUMENT, "srh_mask_host is NULL");
  const int G = p->n_q_heads / p->n_kv_heads;
  ls.off.assign(p->n_kv_heads + 1, 0);
  ls.head.clear();
  ls.nmax = 0;
  for (int g = 0; g < p->n_kv_heads; ++g) {
    int n = 0;
    for (int h = g * G; h < (g + 1) * G; ++h) {
      if (mask[h]) {
        ls.head.push_back((uint8_t)h);
        ++n;
      }
    }
    if (n == 0 && p->index_mode != CKV_INDEX_LAYER)
      return fail(CKV_INVALID_ARGUMENT, "layer %d: KV group %d has no Semantic Retrieval Head",
                  layer, g);
    ls.nmax = std::max(ls.nmax, n);
    ls.off[g + 1] = (uint16_t)ls.head.size();
  }
  if (ls.head.empty())
    return fail(CKV_INVALID_ARGUMENT, "layer %d has no Semantic Retrieval Head", layer);
  return CKV_OK;
}

// Row tiles per SRH, the largest group, and the SRH-end bits of the row tiles.
int set_row_tiles(const ckv_problem *p, int nmax, Plan &pl) {
  pl.th = (p->window + 15) / 16;
  pl.nmax = nmax;
  pl.rt_max = nmax * pl.th;
  // 16 row tiles of fp32 queries at head_dim 128 would not fit the LDS
  const int cap = (p->dtype == CKV_F32 && p->head_dim == 128) ? 12 : 16;
  if (pl.rt_max > cap)
    return fail(CKV_UNSUPPORTED,
                "ceil(window/16) * SRHs per group must be <= %d (window %d, %d SRHs)", cap,
                p->window, nmax);
  pl.head_end_mask = 0;
  for (int rt = 0; rt < 32; ++rt)
    if ((rt + 1) % pl.th == 0) pl.head_end_mask |= 1u << rt;
  return CKV_OK;
}

int check_mask(const ckv_problem *p, const uint8_t *mask, Plan &pl) {
  int st;
  if ((st = layer_srh(p, mask, 0, pl.srh))) return st;
  if ((st = set_row_tiles(p, pl.srh.nmax, pl))) return st;
  pl.rt_layer.assign(1, pl.rt_max);
  return CKV_OK;
}

// Chunk sizes of the two-pass kernels: multiples of 512 keys (statistics: an
// even number of 2-tile groups for each of the 4 waves) and 992 + 32 halo keys
// (column sums: an even number of 2-tile groups for each of the 4 waves).
// Both depend on the layer's shape only.
void set_chunks(const ckv_problem *p, Plan &pl) {
  pl.T = p->cu_seqlens_host[p->batch];
  pl.lmax = 0;
  for (int b = 0; b < p->batch; ++b)
    pl.lmax = std::max(pl.lmax, p->cu_seqlens_host[b + 1] - p->cu_seqlens_host[b]);
  pl.chunk1 = pick_chunk(p, 512, 4096, 256);
  pl.chunk2 = 992;
  pl.max_chunks1 = std::max(1, (pl.lmax + pl.chunk1 - 1) / pl.chunk1);
  pl.max_chunks2 = std::max(1, (pl.lmax + pl.chunk2 - 1) / pl.chunk2);
}

// Workgroups of cpw chunks first, then at least `tail` chunks of every
// (sequence, group) one per workgroup, so the end of each scoring grid is made
// of short workgroups.
void set_lead(Plan &pl, int tail1, int tail2) {
  pl.lead1 = pl.cpw1 > 1 ? std::max(0, (pl.max_chunks1 - tail1) / pl.cpw1) : pl.max_chunks1;
  pl.lead2 = pl.cpw2 > 1 ? std::max(0, (pl.max_chunks2 - tail2) / pl.cpw2) : pl.max_chunks2;
}

// Units of the single-pass kernel in a sequence of L keys.
int op_units(int L) { return (L + ckv::kOnePassUnitKeys - 1) / ckv::kOnePassUnitKeys; }

// Row tiles a layer may have to be scored in a single pass.
constexpr int kOnePassMaxRowTiles = 6;
// Polls of a late normaliser before a unit is left to the catch-up kernel.
constexpr int kDefaultSpinLimit = 64;
// Row tiles per group of the fused two-pass launch, and the polls of a
// group's partials before a workgroup leaves its column sums to catch-up.
constexpr int kFusedMaxRowTiles = 8;
// CKV_SCORE_AUTO takes the one launch up to 6 row tiles: at 8 (the Qwen shape,
// 128 rows per group) two launches measured faster (1.65 against 1.79 ms per
// score phase; there the statistics kernel runs three waves per SIMD, the
// one launch two).
constexpr int kFusedAutoMaxRowTiles = 6;
constexpr int kFusedMinChunks = 16;   // statistics chunks per sequence for CKV_SCORE_AUTO
constexpr int kDefaultFusedSpin = 256;

// Whether the problem's shape allows single-pass scoring at all (bf16 keys,
// per-group selections, a batch that fits the kernel's ticket table); the
// workspace of such problems always has room for it.
bool op_shape(const ckv_problem *p) {
  return p->scoring != CKV_SCORE_TWO_PASS && p->scoring != CKV_SCORE_TWO_LAUNCHES &&
         p->dtype == CKV_BF16 &&
         p->index_mode == CKV_INDEX_PER_GROUP && p->batch <= ckv::kOnePassMaxBatch;
}

// CUs of the current device (0 if the query fails).
int device_cus() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return 0;
  return cus;
}

// Which layers are scored in a single pass, and the table order (those
// layers first).  CKV_SCORE_AUTO picks the two-pass kernels, which are the
// faster of the two on the shapes measured; CKV_SCORE_ONE_PASS asks for the
// single pass on every layer (CKV_UNSUPPORTED where a layer does not
// qualify: more than 6 row tiles in a group).  The choice for a layer depends
// only on the problem and that layer's masks, so multi-layer calls score
// every layer as the single-layer call would.
int choose_paths(const ckv_problem *p, Plan &pl) {
  const int n = pl.n_layers;
  std::vector<uint8_t> op(n, 0);
  pl.op_grid = 0;
  if (pl.op_shape && p->scoring == CKV_SCORE_ONE_PASS)
    for (int l = 0; l < n; ++l) op[l] = pl.rt_layer[l] <= kOnePassMaxRowTiles;
  if (p->scoring == CKV_SCORE_ONE_PASS) {
    if (!pl.op_shape)
      return fail(CKV_UNSUPPORTED, "single-pass scoring needs bf16 inputs, CKV_INDEX_PER_GROUP "
                                   "and batch <= %d", ckv::kOnePassMaxBatch);
    for (int l = 0; l < n; ++l)
      if (!op[l])
        return fail(CKV_UNSUPPORTED, "layer %d: single-pass scoring needs at most %d row tiles "
                                     "per group (ceil(W/16) * SRHs)", l, kOnePassMaxRowTiles);
  }
  pl.order.clear();
  pl.n_op = 0;
  pl.op_rt_max = pl.tp_rt_max = 0;
  for (int l = 0; l < n; ++l)
    if (op[l]) {
      pl.order.push_back(l);
      pl.op_rt_max = std::max(pl.op_rt_max, pl.rt_layer[l]);
    }
  pl.n_op = (int)pl.order.size();
  for (int l = 0; l < n; ++l)
    if (!op[l]) {
      pl.order.push_back(l);
      pl.tp_rt_max = std::max(pl.tp_rt_max, pl.rt_layer[l]);
    }
  if (pl.n_op > 0 && pl.op_grid == 0) pl.op_grid = device_cus();
  if (pl.n_op > 0 && pl.op_grid == 0)
    return fail(CKV_HIP_ERROR, "no HIP device for the single-pass kernel");
  return CKV_OK;
}

// Workspace layout (see Plan).  The counters block and the partial statistics
// of the single-pass layers are contiguous: the single-pass launch zeroes them.
void set_layout(const ckv_problem *p, Plan &pl) {
  const int n = pl.n_layers;
  const size_t groups = (size_t)p->batch * p->n_kv_heads;
  const size_t lg = groups * n;
  pl.op_shape = op_shape(p);
  pl.units_layer = 0;
  for (int b = 0; b < p->batch; ++b)
    pl.units_layer += p->n_kv_heads * op_units(p->cu_seqlens_host[b + 1] - p->cu_seqlens_host[b]);
  pl.ew = p->pool_kernel - 1;
  pl.max_parts = pl.max_chunks1;
  if (pl.op_shape) pl.max_parts = std::max(pl.max_parts, op_units(pl.lmax));
  const int row_slots = pl.rt_max * 16;
  pl.stats_layer = (int64_t)(groups * pl.max_parts * (size_t)row_slots);
  pl.hist_layer = (int64_t)(groups * ckv::kHistBins);
  pl.table_off = 0;
  pl.scores_off = round_up((size_t)n * sizeof(ckv::LayerDesc), 256);
  pl.counters_off = pl.scores_off + round_up((size_t)n * p->n_kv_heads * pl.T * sizeof(float), 256);
  pl.arrive_off = pl.counters_off + 256;
  pl.bias_off = pl.arrive_off + round_up(lg * sizeof(int), 256);
  pl.hist_off = pl.bias_off + round_up(lg * row_slots * sizeof(float2), 256);
  pl.stats_off = pl.hist_off + round_up(lg * ckv::kHistBins * sizeof(int), 256);
  pl.skip_off = pl.stats_off + round_up((size_t)n * pl.stats_layer * sizeof(float2), 256);
  pl.edges_off = pl.skip_off;
  pl.total = pl.skip_off;
  if (pl.op_shape) {
    const size_t units = (size_t)n * pl.units_layer;
    pl.edges_off = pl.skip_off + round_up(units * sizeof(int), 256);
    pl.total = pl.edges_off +
               round_up(units * (size_t)pl.nmax * 2 * pl.ew * sizeof(float), 256);
  }
  // Both passes in one launch where its workgroups fit two to a CU (bf16, at
  // most 8 row tiles per group); the library's own choice also needs every
  // sequence to give most of a group's workgroups a statistics chunk (shorter
  // sequences leave them idle: two launches are faster there, as measured).
  bool long_enough = true;
  for (int b = 0; b < p->batch; ++b)
    long_enough = long_enough && p->cu_seqlens_host[b + 1] - p->cu_seqlens_host[b] >=
                                     kFusedMinChunks * pl.chunk1;
  // (its catch-up list is reserved wherever the shape allows it, so that the
  // workspace size does not depend on the scoring field)
  const bool fused_shape = p->dtype == CKV_BF16 && pl.rt_max <= kFusedMaxRowTiles;
  pl.fused = fused_shape && (p->scoring == CKV_SCORE_TWO_PASS ||
                             (p->scoring == CKV_SCORE_AUTO && long_enough &&
                              pl.rt_max <= kFusedAutoMaxRowTiles));
  if (fused_shape) {
    pl.fskip_off = round_up(pl.total, 256);
    const int64_t nb = ckv::fused_blocks(p->n_kv_heads, p->batch * n);
    pl.total = pl.fskip_off + round_up((size_t)(1 + nb) * sizeof(int), 256);
  }
  // Selections over more than one slice of prefix positions are split over
  // their slices (per-group index sets, whose first digit the column sums
  // count).
  pl.sel_slices = 0;
  const int pmax = pl.lmax - p->window;
  if (p->index_mode == CKV_INDEX_PER_GROUP && pmax > ckv::kSelSlice &&
      pmax <= ckv::kSelSlice * ckv::kMaxSelSlices) {
    const int ns = (pmax + ckv::kSelSlice - 1) / ckv::kSelSlice;
    pl.sel_slices = ns;
    pl.sel_meta_off = round_up(pl.total, 256);
    pl.sel_cand_off = pl.sel_meta_off +
                      round_up(lg * ns * (size_t)ckv::kSelMetaPerSlice * sizeof(int), 256);
    pl.sel_ord_off = pl.sel_cand_off + round_up(lg * ns * (size_t)ckv::kSelSliceCap * 4, 256);
    pl.total = pl.sel_ord_off + round_up(lg * ns * (size_t)ckv::kSelSliceCap * 8, 256);
  }
}

// One-chunk workgroups at the end of the multi-layer scoring grids, per
// (sequence, group) and layer.
constexpr int kTail1 = 4, kTail2 = 4;

// The plan of a call over n_layers layers (rt_layer set): chunking, grid
// shapes and workspace layout; with decide_path also the scoring path of
// every layer (may query the device, may fail with CKV_UNSUPPORTED).
int make_plan(const ckv_problem *p, int n_layers, Plan &pl, bool decide_path) {
  set_chunks(p, pl);
  pl.n_layers = n_layers;
  if (n_layers > 1) {
    // Longer workgroups once there are enough of them: a few rounds of the
    // resident workgroups keep the tail short, and every round keeps its key
    // stream going across chunk boundaries.
    const int64_t units1 = (int64_t)p->batch * p->n_kv_heads * n_layers * pl.max_chunks1;
    const int64_t units2 = (int64_t)p->batch * p->n_kv_heads * n_layers * pl.max_chunks2;
    pl.cpw1 = (int)std::max<int64_t>(1, std::min<int64_t>(8, units1 / 3072));
    pl.cpw2 = (int)std::max<int64_t>(1, std::min<int64_t>(8, units2 / 2048));
    set_lead(pl, kTail1, kTail2);
  } else {
    pl.cpw1 = pl.cpw2 = 1;
    set_lead(pl, 0, 0);
  }
  set_layout(p, pl);
  if (!decide_path) return CKV_OK;
  return choose_paths(p, pl);
}

// Fields of the scoring arguments shared by every layer.
ckv::ScoreArgs score_args(const ckv_problem *p, const Plan &pl, void *ws) {
  ckv::ScoreArgs a{};
  a.layers = nullptr;
  a.cu = p->cu_seqlens;
  a.stats = reinterpret_cast<float2 *>(static_cast<char *>(ws) + pl.stats_off);
  a.stats_layer = pl.stats_layer;
  a.hist = reinterpret_cast<int *>(static_cast<char *>(ws) + pl.hist_off);
  a.hist_layer = pl.hist_layer;
  a.k_stride_tok = p->k_stride_tok;
  a.k_stride_head = p->k_stride_head;
  a.T = (int32_t)pl.T;
  a.batch = p->batch;
  a.Hq = p->n_q_heads;
  a.Hkv = p->n_kv_heads;
  a.W = p->window;
  a.th = pl.th;
  a.row_slots = pl.rt_max * 16;   // partial and normaliser slots per group
  a.chunk1 = pl.chunk1;
  a.max_chunks1 = pl.max_chunks1;
  a.parts_stride = pl.max_parts;   // partial slots between groups
  a.cpw1 = pl.cpw1;
  a.cpw2 = pl.cpw2;
  a.lead1 = pl.lead1;
  a.lead2 = pl.lead2;
  a.nz = 0;   // set by the launcher
  a.chunk2 = pl.chunk2;
  a.max_chunks2 = pl.max_chunks2;
  const double scale = p->scale > 0.f ? (double)p->scale : 1.0 / std::sqrt((double)p->head_dim);
  a.c1 = (float)(scale * 1.4426950408889634);
  a.pool_kernel = p->pool_kernel;
  a.pool_type = p->pool_type;
  a.reduce_order = p->reduce_order;
  a.head_end_mask = pl.head_end_mask;
  a.fused_skip =
      pl.fused ? reinterpret_cast<int *>(static_cast<char *>(ws) + pl.fskip_off) : nullptr;
  a.fused_arrive = reinterpret_cast<int *>(static_cast<char *>(ws) + pl.arrive_off);
  a.fused_bias = reinterpret_cast<float2 *>(static_cast<char *>(ws) + pl.bias_off);
  a.fused_spin = p->spin_limit == CKV_SPIN_CATCHUP_ALL ? -1
                 : p->spin_limit < 0                 ? kDefaultFusedSpin
                                                     : p->spin_limit;
  return a;
}

// The inline layer of a single-layer call.
ckv::LayerDesc layer_desc(const LayerSrh *srh, const void *q, const void *k, const void *v,
                          float *scores, int32_t *idx, void *k_out, void *v_out, int32_t budget) {
  ckv::LayerDesc d{};
  d.q = q;
  d.k = k;
  d.v = v;
  d.scores = scores;
  d.idx = idx;
  d.k_out = k_out;
  d.v_out = v_out;
  d.budget = budget;
  if (srh) {
    for (size_t i = 0; i < srh->off.size(); ++i) d.srh_off[i] = srh->off[i];
    for (size_t i = 0; i < srh->head.size(); ++i) d.srh_head[i] = srh->head[i];
  }
  return d;
}

int check_ptr(const void *ptr, const char *name, size_t align) {
  if (!ptr) return fail(CKV_INVALID_ARGUMENT, "%s is NULL", name);
  if (!aligned(ptr, align)) return fail(CKV_UNSUPPORTED, "%s must be %zu-byte aligned", name, align);
  return CKV_OK;
}

int check_budget(const ckv_problem *p, int32_t budget) {
  if (budget < p->window)
    return fail(CKV_INVALID_ARGUMENT, "budget (%d) must be >= window (%d)", budget, p->window);
  return CKV_OK;
}

int check_ws(const Plan &pl, const void *ws, size_t ws_bytes) {
  if (ws_bytes < pl.total)
    return fail(CKV_WORKSPACE_TOO_SMALL, "workspace of %zu bytes, %zu needed", ws_bytes, pl.total);
  if (pl.total > 0) {
    if (!ws) return fail(CKV_INVALID_ARGUMENT, "workspace is NULL");
    if (!aligned(ws, 256)) return fail(CKV_UNSUPPORTED, "workspace must be 256-byte aligned");
  }
  return CKV_OK;
}

int hip_status(hipError_t e, const char *what) {
  if (e != hipSuccess)
    return fail(CKV_HIP_ERROR, "%s launch failed: %s", what, hipGetErrorString(e));
  return CKV_OK;
}

// ws: the call's workspace (NULL: no split selection).
ckv::SelectArgs select_args(const ckv_problem *p, const Plan &pl, const int *hist, void *ws) {
  ckv::SelectArgs s{};
  s.layers = nullptr;
  s.hist = hist;
  s.hist_layer = pl.hist_layer;
  s.cu = p->cu_seqlens;
  s.T = (int32_t)pl.T;
  s.Hkv = p->n_kv_heads;
  s.W = p->window;
  s.batch = p->batch;
  const bool shared = p->index_mode == CKV_INDEX_LAYER;
  s.n_sel = shared ? 1 : p->n_kv_heads;
  s.out_groups = shared ? p->n_kv_heads : 1;
  if (shared) s.hist = nullptr;   // the histograms are per group: count the layer score
  if (pl.sel_slices > 0 && s.hist && ws) {
    s.sel_meta = reinterpret_cast<int *>(static_cast<char *>(ws) + pl.sel_meta_off);
    s.sel_cand = reinterpret_cast<uint32_t *>(static_cast<char *>(ws) + pl.sel_cand_off);
    s.sel_ord = reinterpret_cast<uint64_t *>(static_cast<char *>(ws) + pl.sel_ord_off);
    s.n_slices = pl.sel_slices;
    s.cand_cap = ckv::kSelSliceCap;
  }
  return s;
}

// Layer-shared index set: the layer score into every group's row.
hipError_t launch_combine_if_shared(const ckv_problem *p, const Plan &pl, const LayerSrh *srh,
                                    float *scores, const ckv::LayerDesc *table, int n_layers,
                                    hipStream_t stream) {
  if (p->index_mode != CKV_INDEX_LAYER) return hipSuccess;
  ckv::CombineArgs c{};
  if (srh) c.l0 = layer_desc(srh, nullptr, nullptr, nullptr, scores, nullptr, nullptr, nullptr, 0);
  c.layers = table;
  c.cu = p->cu_seqlens;
  c.T = (int32_t)pl.T;
  c.Hkv = p->n_kv_heads;
  c.W = p->window;
  c.batch = p->batch;
  return ckv::launch_combine(c, n_layers, pl.lmax, stream);
}

ckv::GatherArgs gather_args(const ckv_problem *p) {
  const int es = elem_size(p);
  ckv::GatherArgs g{};
  g.layers = nullptr;
  g.cu = p->cu_seqlens;
  g.k_stride_tok = p->k_stride_tok * es;
  g.k_stride_head = p->k_stride_head * es;
  g.v_stride_tok = p->v_stride_tok * es;
  g.v_stride_head = p->v_stride_head * es;
  g.Hkv = p->n_kv_heads;
  g.batch = p->batch;
  g.row_bytes = p->head_dim * es;
  return g;
}

// Host-side arrays of a multi-layer call (entries may be NULL where the call
// does not use them).
struct LayerPtrs {
  const void *const *q = nullptr, *const *k = nullptr, *const *v = nullptr;
  int32_t *const *idx = nullptr;
  void *const *k_out = nullptr, *const *v_out = nullptr;
  const int32_t *budgets = nullptr;
};

// Validation of a multi-layer call: every layer's SRH mask (-> pl.rt_max) and,
// where given, its budget and pointers.
int check_layers(const ckv_problem *p, int n_layers, const uint8_t *masks, const LayerPtrs &lp,
                 Plan &pl, std::vector<uint32_t> *bits) {
  if (n_layers < 1) return fail(CKV_INVALID_ARGUMENT, "n_layers must be >= 1 (got %d)", n_layers);
  if ((int64_t)n_layers * p->batch > 65535)
    return fail(CKV_UNSUPPORTED, "n_layers * batch must be <= 65535");
  if (!masks) return fail(CKV_INVALID_ARGUMENT, "srh_masks_host is NULL");
  int nmax = 0, st;
  LayerSrh ls;
  std::vector<int> nmax_layer(n_layers);
  if (bits) bits->assign((size_t)n_layers * (ckv::kMaxQHeads / 32), 0u);
  for (int l = 0; l < n_layers; ++l) {
    const uint8_t *m = masks + (size_t)l * p->n_q_heads;
    if ((st = layer_srh(p, m, l, ls))) return st;
    nmax = std::max(nmax, ls.nmax);
    nmax_layer[l] = ls.nmax;
    if (bits)
      for (int h = 0; h < p->n_q_heads; ++h)
        if (m[h]) (*bits)[(size_t)l * (ckv::kMaxQHeads / 32) + h / 32] |= 1u << (h % 32);
  }
  if ((st = set_row_tiles(p, nmax, pl))) return st;
  pl.rt_layer.resize(n_layers);
  for (int l = 0; l < n_layers; ++l) pl.rt_layer[l] = nmax_layer[l] * pl.th;
  char name[64];
  for (int l = 0; l < n_layers; ++l) {
    if (lp.budgets) {
      if (lp.budgets[l] < p->window)
        return fail(CKV_INVALID_ARGUMENT, "layer %d: budget (%d) must be >= window (%d)", l,
                    lp.budgets[l], p->window);
    }
    struct {
      const void *ptr;
      const char *what;
      size_t align;
    } checks[] = {{lp.q ? lp.q[l] : nullptr, "q_win", 16}, {lp.k ? lp.k[l] : nullptr, "k", 16},
                  {lp.v ? lp.v[l] : nullptr, "v", 16},     {lp.idx ? lp.idx[l] : nullptr, "idx", 4},
                  {lp.k_out ? lp.k_out[l] : nullptr, "k_out", 16},
                  {lp.v_out ? lp.v_out[l] : nullptr, "v_out", 16}};
    const void *const *arrays[] = {(const void *const *)lp.q, (const void *const *)lp.k,
                                   (const void *const *)lp.v, (const void *const *)lp.idx,
                                   (const void *const *)lp.k_out, (const void *const *)lp.v_out};
    for (int i = 0; i < 6; ++i) {
      if (!arrays[i]) continue;   // not used by this call
      snprintf(name, sizeof name, "layer %d: %s", l, checks[i].what);
      if ((st = check_ptr(checks[i].ptr, name, checks[i].align))) return st;
    }
  }
  return CKV_OK;
}

// Enqueue the writes of the layer table: entry i describes the caller's layer
// pl.order[i] (its scores at scores + that layer's slice).
hipError_t put_layers(const ckv_problem *p, const Plan &pl, const LayerPtrs &lp,
                      const std::vector<uint32_t> &bits, float *scores, void *ws,
                      hipStream_t stream) {
  ckv::LayerDesc *table =
      reinterpret_cast<ckv::LayerDesc *>(static_cast<char *>(ws) + pl.table_off);
  const size_t per_layer_scores = (size_t)p->n_kv_heads * pl.T;
  const int n_layers = pl.n_layers;
  for (int first = 0; first < n_layers; first += ckv::kPutLayers) {
    ckv::PutArgs a{};
    a.table = table;
    a.first = first;
    a.count = std::min(ckv::kPutLayers, n_layers - first);
    a.Hq = p->n_q_heads;
    a.Hkv = p->n_kv_heads;
    for (int i = 0; i < a.count; ++i) {
      const int l = pl.order[first + i];
      ckv::PutEntry &e = a.e[i];
      e.q = lp.q ? lp.q[l] : nullptr;
      e.k = lp.k ? lp.k[l] : nullptr;
      e.v = lp.v ? lp.v[l] : nullptr;
      e.scores = scores + (size_t)l * per_layer_scores;
      e.idx = lp.idx ? lp.idx[l] : nullptr;
      e.k_out = lp.k_out ? lp.k_out[l] : nullptr;
      e.v_out = lp.v_out ? lp.v_out[l] : nullptr;
      e.budget = lp.budgets ? lp.budgets[l] : 0;
      for (int w = 0; w < ckv::kMaxQHeads / 32; ++w)
        e.srh_bits[w] = bits[(size_t)l * (ckv::kMaxQHeads / 32) + w];
    }
    hipError_t err = ckv::launch_put_layers(a, stream);
    if (err != hipSuccess) return err;
  }
  return hipSuccess;
}

// The single-pass kernels over table entries 0 .. n_op - 1.
hipError_t launch_onepass(const ckv_problem *p, const Plan &pl, const ckv::ScoreArgs &a,
                          void *ws, hipStream_t stream) {
  ckv::OnePassArgs f{};
  f.s = a;
  char *w = static_cast<char *>(ws);
  f.fill_base = reinterpret_cast<int *>(w + pl.counters_off);
  f.ticket = f.fill_base;
  f.skip_count = f.fill_base + 1;
  f.arrive = reinterpret_cast<int *>(w + pl.arrive_off);
  f.bias = reinterpret_cast<float2 *>(w + pl.bias_off);
  f.skip_list = reinterpret_cast<int *>(w + pl.skip_off);
  f.edges = reinterpret_cast<float *>(w + pl.edges_off);
  int acc = 0;
  for (int b = 0; b <= p->batch; ++b) {
    f.seq_units[b] = acc;
    if (b < p->batch)
      acc += p->n_kv_heads * op_units(p->cu_seqlens_host[b + 1] - p->cu_seqlens_host[b]);
  }
  f.units_per_layer = acc;
  f.n_units_total = acc * pl.n_op;
  f.spin_limit = p->spin_limit == CKV_SPIN_CATCHUP_ALL ? -1
                 : p->spin_limit < 0                 ? kDefaultSpinLimit
                                                     : p->spin_limit;
  f.ew = pl.ew;
  f.heads_max = pl.nmax;
  const size_t fill_end = pl.stats_off + (size_t)pl.n_op * pl.stats_layer * sizeof(float2);
  const int64_t fill_ints = (int64_t)((fill_end - pl.counters_off) / sizeof(int));
  return ckv::launch_onepass(f, p->head_dim, pl.op_rt_max, pl.op_grid, fill_ints, stream);
}

// The two-pass kernels over table entries n_op .. n_layers - 1.
hipError_t launch_twopass_table(const ckv_problem *p, const Plan &pl, const ckv::ScoreArgs &a,
                                hipStream_t stream) {
  const int n_tp = pl.n_layers - pl.n_op;
  if (n_tp == 0) return hipSuccess;
  ckv::ScoreArgs b = a;
  b.layers = a.layers + pl.n_op;
  b.stats = a.stats + pl.n_op * a.stats_layer;
  b.hist = a.hist + pl.n_op * a.hist_layer;
  const int64_t groups = (int64_t)p->batch * p->n_kv_heads;
  b.fused_arrive = a.fused_arrive + pl.n_op * groups;
  b.fused_bias = a.fused_bias + pl.n_op * groups * a.row_slots;
  return ckv::launch_score_layers(b, p->dtype == CKV_BF16, p->head_dim, pl.tp_rt_max, p->batch,
                                  n_tp, stream);
}

// S1-S4 of a single-layer call on the path the plan chose.
hipError_t launch_scoring(const ckv_problem *p, const Plan &pl, const void *q, const void *k,
                          float *scores, void *ws, hipStream_t stream) {
  ckv::ScoreArgs a = score_args(p, pl, ws);
  if (pl.n_op == 0) {
    a.l0 = layer_desc(&pl.srh, q, k, nullptr, scores, nullptr, nullptr, nullptr, 0);
    return ckv::launch_score(a, p->dtype == CKV_BF16, p->head_dim, pl.rt_max, p->batch, stream);
  }
  // the single-pass kernel reads its operands from a layer table
  LayerPtrs lp;
  lp.q = &q;
  lp.k = &k;
  std::vector<uint32_t> bits(ckv::kMaxQHeads / 32, 0u);
  for (uint8_t h : pl.srh.head) bits[h / 32] |= 1u << (h % 32);
  hipError_t e = put_layers(p, pl, lp, bits, scores, ws, stream);
  if (e != hipSuccess) return e;
  a.layers = reinterpret_cast<const ckv::LayerDesc *>(static_cast<char *>(ws) + pl.table_off);
  return launch_onepass(p, pl, a, ws, stream);
}

// S1-S4 (and, with budgets, S5-S6) of a multi-layer call.
int run_layers(const ckv_problem *p, int n_layers, const LayerPtrs &lp, const uint8_t *masks,
               float *scores_or_null, void *ws, size_t ws_bytes, void *stream, bool full) {
  Plan pl;
  std::vector<uint32_t> bits;
  int st;
  if ((st = check_problem(p))) return st;
  if ((st = check_layers(p, n_layers, masks, lp, pl, &bits))) return st;
  if (!full && (st = check_ptr(scores_or_null, "scores", 4))) return st;
  if (scores_or_null && (st = check_ptr(scores_or_null, "scores", 4))) return st;
  make_plan(p, n_layers, pl, false);
  if ((st = check_ws(pl, ws, ws_bytes))) return st;
  if ((st = make_plan(p, n_layers, pl, true))) return st;
  float *scores = scores_or_null
                      ? scores_or_null
                      : reinterpret_cast<float *>(static_cast<char *>(ws) + pl.scores_off);
  hipStream_t s = (hipStream_t)stream;
  if ((st = hip_status(put_layers(p, pl, lp, bits, scores, ws, s), "layer table"))) return st;
  const ckv::LayerDesc *table =
      reinterpret_cast<const ckv::LayerDesc *>(static_cast<char *>(ws) + pl.table_off);
  ckv::ScoreArgs a = score_args(p, pl, ws);
  a.layers = table;
  if (pl.n_op > 0 && (st = hip_status(launch_onepass(p, pl, a, ws, s), "score"))) return st;
  if ((st = hip_status(launch_twopass_table(p, pl, a, s), "score"))) return st;
  if ((st = hip_status(launch_combine_if_shared(p, pl, nullptr, nullptr, table, n_layers, s),
                       "combine")))
    return st;
  if (!full) return ok();
  ckv::SelectArgs sa = select_args(p, pl, a.hist, ws);
  sa.layers = table;
  if ((st = hip_status(ckv::launch_select(sa, n_layers, s), "select"))) return st;
  ckv::GatherArgs ga = gather_args(p);
  ga.layers = table;
  int max_budget = 0;
  for (int l = 0; l < n_layers; ++l) max_budget = std::max(max_budget, lp.budgets[l]);
  if ((st = hip_status(ckv::launch_gather(ga, n_layers, max_budget, s), "gather"))) return st;
  return ok();
}

// Per-group budgets from the host array (head-level allocation).
int check_group_budgets(const ckv_problem *p, const int32_t *gb_host, ckv::GroupBudgets &gb,
                        int *max_budget) {
  if (!gb_host) return fail(CKV_INVALID_ARGUMENT, "group_budgets_host is NULL");
  if (p->index_mode == CKV_INDEX_LAYER)
    return fail(CKV_UNSUPPORTED, "per-group budgets need per-group selections "
                                 "(CKV_INDEX_PER_GROUP)");
  int64_t total = 0;
  *max_budget = 0;
  gb = ckv::GroupBudgets{};
  for (int g = 0; g < p->n_kv_heads; ++g) {
    if (gb_host[g] < p->window)
      return fail(CKV_INVALID_ARGUMENT, "group %d: budget (%d) must be >= window (%d)", g,
                  gb_host[g], p->window);
    gb.budget[g] = gb_host[g];
    gb.off[g] = (int32_t)total;
    total += gb_host[g];
    *max_budget = std::max(*max_budget, gb_host[g]);
  }
  if (total * p->batch > INT32_MAX)
    return fail(CKV_UNSUPPORTED, "batch * sum of the group budgets must fit in int32");
  gb.on = 1;
  gb.total = (int32_t)total;
  return CKV_OK;
}

}  // namespace

extern "C" {

const char *compresskv_status_string(int status) {
  switch (status) {
    case CKV_OK: return "ok";
    case CKV_INVALID_ARGUMENT: return "invalid argument";
    case CKV_UNSUPPORTED: return "unsupported";
    case CKV_WORKSPACE_TOO_SMALL: return "workspace too small";
    case CKV_HIP_ERROR: return "HIP error";
    default: return "unknown status";
  }
}

const char *compresskv_last_error(void) { return g_last_error.c_str(); }

int compresskv_scoring_path(const ckv_problem *p, const uint8_t *srh_mask_host) {
  Plan pl;
  int st;
  if ((st = check_problem(p))) return -st;
  if ((st = check_mask(p, srh_mask_host, pl))) return -st;
  if ((st = make_plan(p, 1, pl, true))) return -st;
  ok();
  return pl.n_op > 0 ? 1 : pl.fused ? 3 : 2;
}

size_t compresskv_workspace_bytes(const ckv_problem *p, const uint8_t *srh_mask_host,
                                  int32_t budget) {
  Plan pl;
  if (check_problem(p) || check_mask(p, srh_mask_host, pl) || check_budget(p, budget)) return 0;
  make_plan(p, 1, pl, false);
  ok();
  return pl.total;
}

int compresskv_score(const ckv_problem *p, const void *q_win, const void *k,
                     const uint8_t *srh_mask_host, float *scores, void *ws, size_t ws_bytes,
                     void *stream) {
  Plan pl;
  int st;
  if ((st = check_problem(p))) return st;
  if ((st = check_mask(p, srh_mask_host, pl))) return st;
  if ((st = check_ptr(q_win, "q_win", 16)) || (st = check_ptr(k, "k", 16)) ||
      (st = check_ptr(scores, "scores", 4)))
    return st;
  make_plan(p, 1, pl, false);
  if ((st = check_ws(pl, ws, ws_bytes))) return st;
  if ((st = make_plan(p, 1, pl, true))) return st;
  if ((st = hip_status(launch_scoring(p, pl, q_win, k, scores, ws, (hipStream_t)stream),
                       "score")))
    return st;
  if ((st = hip_status(
           launch_combine_if_shared(p, pl, &pl.srh, scores, nullptr, 0, (hipStream_t)stream),
           "combine")))
    return st;
  return ok();
}

int compresskv_select(const ckv_problem *p, const float *scores, int32_t budget, int32_t *idx,
                      void *ws, size_t ws_bytes, void *stream) {
  (void)ws;
  (void)ws_bytes;
  int st;
  if ((st = check_problem(p))) return st;
  if ((st = check_budget(p, budget))) return st;
  if ((st = check_ptr(scores, "scores", 4)) || (st = check_ptr(idx, "idx", 4))) return st;
  Plan pl;
  pl.T = p->cu_seqlens_host[p->batch];
  ckv::SelectArgs sa = select_args(p, pl, nullptr, nullptr);
  sa.l0 = layer_desc(nullptr, nullptr, nullptr, nullptr, const_cast<float *>(scores), idx,
                     nullptr, nullptr, budget);
  if ((st = hip_status(ckv::launch_select(sa, 0, (hipStream_t)stream), "select"))) return st;
  return ok();
}

int compresskv_gather(const ckv_problem *p, const void *k, const void *v, const int32_t *idx,
                      int32_t budget, void *k_out, void *v_out, void *stream) {
  int st;
  if ((st = check_problem(p))) return st;
  if (budget < 1) return fail(CKV_INVALID_ARGUMENT, "budget must be >= 1 (got %d)", budget);
  if ((st = check_ptr(k, "k", 16)) || (st = check_ptr(v, "v", 16)) ||
      (st = check_ptr(idx, "idx", 4)) || (st = check_ptr(k_out, "k_out", 16)) ||
      (st = check_ptr(v_out, "v_out", 16)))
    return st;
  ckv::GatherArgs ga = gather_args(p);
  ga.l0 = layer_desc(nullptr, nullptr, k, v, nullptr, const_cast<int32_t *>(idx), k_out, v_out,
                     budget);
  if ((st = hip_status(ckv::launch_gather(ga, 0, budget, (hipStream_t)stream), "gather")))
    return st;
  return ok();
}

int compresskv_compress_layer(const ckv_problem *p, const void *q_win, const void *k,
                              const void *v, const uint8_t *srh_mask_host, int32_t budget,
                              int32_t *idx, void *k_out, void *v_out, float *scores_or_null,
                              void *ws, size_t ws_bytes, void *stream) {
  Plan pl;
  int st;
  if ((st = check_problem(p))) return st;
  if ((st = check_mask(p, srh_mask_host, pl))) return st;
  if ((st = check_budget(p, budget))) return st;
  if ((st = check_ptr(q_win, "q_win", 16)) || (st = check_ptr(k, "k", 16)) ||
      (st = check_ptr(v, "v", 16)) || (st = check_ptr(idx, "idx", 4)) ||
      (st = check_ptr(k_out, "k_out", 16)) || (st = check_ptr(v_out, "v_out", 16)))
    return st;
  if (scores_or_null && (st = check_ptr(scores_or_null, "scores", 4))) return st;
  make_plan(p, 1, pl, false);
  if ((st = check_ws(pl, ws, ws_bytes))) return st;
  if ((st = make_plan(p, 1, pl, true))) return st;
  float *scores = scores_or_null
                      ? scores_or_null
                      : reinterpret_cast<float *>(static_cast<char *>(ws) + pl.scores_off);
  hipStream_t s = (hipStream_t)stream;
  if ((st = hip_status(launch_scoring(p, pl, q_win, k, scores, ws, s), "score"))) return st;
  if ((st = hip_status(launch_combine_if_shared(p, pl, &pl.srh, scores, nullptr, 0, s),
                       "combine")))
    return st;
  const int *hist = reinterpret_cast<const int *>(static_cast<char *>(ws) + pl.hist_off);
  ckv::SelectArgs sa = select_args(p, pl, hist, ws);
  sa.l0 = layer_desc(nullptr, nullptr, nullptr, nullptr, scores, idx, nullptr, nullptr, budget);
  if ((st = hip_status(ckv::launch_select(sa, 0, s), "select"))) return st;
  ckv::GatherArgs ga = gather_args(p);
  ga.l0 = layer_desc(nullptr, nullptr, k, v, nullptr, idx, k_out, v_out, budget);
  if ((st = hip_status(ckv::launch_gather(ga, 0, budget, s), "gather"))) return st;
  return ok();
}

}  // extern "C"

namespace {

// Scratch of compresskv_compress_layer_noalloc: one array per device, kept
// until the process ends.  In host code `scratch` names a host-side stand-in;
// its device address comes from hipGetSymbolAddress, once per device, with
// that device current.
constexpr size_t kScratchBytes = 32u << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices];

// The current device's scratch address (nullptr and a failure message if the
// lookup fails).
void *device_scratch() {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) {
    fail(CKV_HIP_ERROR, "hipGetDevice failed: %s", hipGetErrorString(e));
    return nullptr;
  }
  if (dev < 0 || dev >= kMaxDevices) {
    fail(CKV_UNSUPPORTED, "device %d: at most %d devices", dev, kMaxDevices);
    return nullptr;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *ptr = nullptr;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr) {
      fail(CKV_HIP_ERROR, "hipGetSymbolAddress(scratch) failed: %s", hipGetErrorString(e));
      return nullptr;
    }
    g_scratch_ptr[dev] = ptr;
  }
  return g_scratch_ptr[dev];
}

}  // namespace

extern "C" {

int compresskv_compress_layer_noalloc(const ckv_problem *p, const void *q_win, const void *k,
                                      const void *v, const uint8_t *srh_mask_host,
                                      int32_t budget, int32_t *idx, void *k_out, void *v_out,
                                      float *scores_or_null, void *stream) {
  Plan pl;
  int st;
  if ((st = check_problem(p))) return st;
  if ((st = check_mask(p, srh_mask_host, pl))) return st;
  if ((st = check_budget(p, budget))) return st;
  make_plan(p, 1, pl, false);
  if (pl.total > kScratchBytes)
    return fail(CKV_WORKSPACE_TOO_SMALL,
                "the problem needs %zu bytes of scratch; the allocation-free entry point has "
                "%zu (use compresskv_compress_layer with a workspace)",
                pl.total, kScratchBytes);
  void *ws = device_scratch();
  if (!ws) return CKV_HIP_ERROR;
  return compresskv_compress_layer(p, q_win, k, v, srh_mask_host, budget, idx, k_out, v_out,
                                   scores_or_null, ws, kScratchBytes, stream);
}

size_t compresskv_layers_workspace_bytes(const ckv_problem *p, int32_t n_layers,
                                         const uint8_t *srh_masks_host) {
  Plan pl;
  if (check_problem(p) || check_layers(p, n_layers, srh_masks_host, LayerPtrs{}, pl, nullptr))
    return 0;
  make_plan(p, n_layers, pl, false);
  ok();
  return pl.total;
}

int compresskv_score_layers(const ckv_problem *p, int32_t n_layers,
                            const void *const *q_win_ptrs_host, const void *const *k_ptrs_host,
                            const uint8_t *srh_masks_host, float *scores, void *ws,
                            size_t ws_bytes, void *stream) {
  LayerPtrs lp;
  if (!q_win_ptrs_host || !k_ptrs_host)
    return fail(CKV_INVALID_ARGUMENT, "q_win_ptrs_host and k_ptrs_host are required");
  lp.q = q_win_ptrs_host;
  lp.k = k_ptrs_host;
  return run_layers(p, n_layers, lp, srh_masks_host, scores, ws, ws_bytes, stream, false);
}

int compresskv_compress_layers(const ckv_problem *p, int32_t n_layers,
                               const void *const *q_win_ptrs_host, const void *const *k_ptrs_host,
                               const void *const *v_ptrs_host, const uint8_t *srh_masks_host,
                               const int32_t *budgets_host, int32_t *const *idx_ptrs_host,
                               void *const *k_out_ptrs_host, void *const *v_out_ptrs_host,
                               float *scores_or_null, void *ws, size_t ws_bytes, void *stream) {
  if (!q_win_ptrs_host || !k_ptrs_host || !v_ptrs_host || !budgets_host || !idx_ptrs_host ||
      !k_out_ptrs_host || !v_out_ptrs_host)
    return fail(CKV_INVALID_ARGUMENT, "every per-layer host array is required");
  LayerPtrs lp;
  lp.q = q_win_ptrs_host;
  lp.k = k_ptrs_host;
  lp.v = v_ptrs_host;
  lp.idx = idx_ptrs_host;
  lp.k_out = k_out_ptrs_host;
  lp.v_out = v_out_ptrs_host;
  lp.budgets = budgets_host;
  return run_layers(p, n_layers, lp, srh_masks_host, scores_or_null, ws, ws_bytes, stream, true);
}

int compresskv_select_heads(const ckv_problem *p, const float *scores,
                            const int32_t *group_budgets_host, int32_t *idx, void *stream) {
  int st, max_budget;
  ckv::GroupBudgets gb;
  if ((st = check_problem(p))) return st;
  if ((st = check_group_budgets(p, group_budgets_host, gb, &max_budget))) return st;
  if ((st = check_ptr(scores, "scores", 4)) || (st = check_ptr(idx, "idx", 4))) return st;
  Plan pl;
  pl.T = p->cu_seqlens_host[p->batch];
  ckv::SelectArgs sa = select_args(p, pl, nullptr, nullptr);
  sa.gb = gb;
  sa.l0 = layer_desc(nullptr, nullptr, nullptr, nullptr, const_cast<float *>(scores), idx,
                     nullptr, nullptr, max_budget);
  if ((st = hip_status(ckv::launch_select(sa, 0, (hipStream_t)stream), "select"))) return st;
  return ok();
}

int compresskv_gather_heads(const ckv_problem *p, const void *k, const void *v,
                            const int32_t *idx, const int32_t *group_budgets_host, void *k_out,
                            void *v_out, void *stream) {
  int st, max_budget;
  ckv::GroupBudgets gb;
  if ((st = check_problem(p))) return st;
  if ((st = check_group_budgets(p, group_budgets_host, gb, &max_budget))) return st;
  if ((st = check_ptr(k, "k", 16)) || (st = check_ptr(v, "v", 16)) ||
      (st = check_ptr(idx, "idx", 4)) || (st = check_ptr(k_out, "k_out", 16)) ||
      (st = check_ptr(v_out, "v_out", 16)))
    return st;
  ckv::GatherArgs ga = gather_args(p);
  ga.gb = gb;
  ga.l0 = layer_desc(nullptr, nullptr, k, v, nullptr, const_cast<int32_t *>(idx), k_out, v_out,
                     max_budget);
  if ((st = hip_status(ckv::launch_gather(ga, 0, max_budget, (hipStream_t)stream), "gather")))
    return st;
  return ok();
}

int compresskv_compress_layer_heads(const ckv_problem *p, const void *q_win, const void *k,
                                    const void *v, const uint8_t *srh_mask_host,
                                    const int32_t *group_budgets_host, int32_t *idx, void *k_out,
                                    void *v_out, float *scores_or_null, void *ws, size_t ws_bytes,
                                    void *stream) {
  Plan pl;
  int st, max_budget;
  ckv::GroupBudgets gb;
  if ((st = check_problem(p))) return st;
  if ((st = check_mask(p, srh_mask_host, pl))) return st;
  if ((st = check_group_budgets(p, group_budgets_host, gb, &max_budget))) return st;
  if ((st = check_ptr(q_win, "q_win", 16)) || (st = check_ptr(k, "k", 16)) ||
      (st = check_ptr(v, "v", 16)) || (st = check_ptr(idx, "idx", 4)) ||
      (st = check_ptr(k_out, "k_out", 16)) || (st = check_ptr(v_out, "v_out", 16)))
    return st;
  if (scores_or_null && (st = check_ptr(scores_or_null, "scores", 4))) return st;
  make_plan(p, 1, pl, false);
  if ((st = check_ws(pl, ws, ws_bytes))) return st;
  if ((st = make_plan(p, 1, pl, true))) return st;
  float *scores = scores_or_null
                      ? scores_or_null
                      : reinterpret_cast<float *>(static_cast<char *>(ws) + pl.scores_off);
  hipStream_t s = (hipStream_t)stream;
  if ((st = hip_status(launch_scoring(p, pl, q_win, k, scores, ws, s), "score"))) return st;
  const int *hist = reinterpret_cast<const int *>(static_cast<char *>(ws) + pl.hist_off);
  ckv::SelectArgs sa = select_args(p, pl, hist, ws);
  sa.gb = gb;
  sa.l0 = layer_desc(nullptr, nullptr, nullptr, nullptr, scores, idx, nullptr, nullptr,
                     max_budget);
  if ((st = hip_status(ckv::launch_select(sa, 0, s), "select"))) return st;
  ckv::GatherArgs ga = gather_args(p);
  ga.gb = gb;
  ga.l0 = layer_desc(nullptr, nullptr, k, v, nullptr, idx, k_out, v_out, max_budget);
  if ((st = hip_status(ckv::launch_gather(ga, 0, max_budget, s), "gather"))) return st;
  return ok();
}

}  // extern "C"
