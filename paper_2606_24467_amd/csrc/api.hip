// C ABI of libcompresskv: host-side validation, workspace layout and dispatch.
// Every check runs before the first HIP call, so invalid arguments never touch
// the device and can be tested without a GPU.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
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

// Everything derived from a validated problem.
struct Plan {
  int64_t T = 0;
  int lmax = 0;
  int n_layers = 1;    // layers of a multi-layer call (1 otherwise)
  int th = 0;          // row tiles per SRH
  int rt_max = 0;      // max row tiles of a group (over the layers)
  int chunk1 = 0, max_chunks1 = 0;
  int chunk2 = 0, max_chunks2 = 0;
  int cpw1 = 1, cpw2 = 1;  // consecutive chunks per leading scoring workgroup
  int lead1 = 1, lead2 = 1;  // leading workgroups per (sequence, group) and layer
  uint32_t head_end_mask = 0;
  // single-layer workspace: scores | stats | counters | histograms
  // multi-layer workspace:  table | scores | stats | histograms (all per layer)
  size_t table_off = 0, scores_off = 0, stats_off = 0, counters_off = 0, bias_off = 0,
         hist_off = 0, total = 0;
  int64_t stats_layer = 0, hist_layer = 0;   // elements per layer
  bool fused = false;      // single-pass scoring kernel
  int n_units_max = 0;     // its units per (sequence, group), largest
  int fused_grid = 0;      // its persistent workgroups
  int n_counters = 0;      // ints zeroed before it (ticket, fallbacks, arrivals,
                           // published normalisers, histograms)
  int max_parts = 0;       // partial-statistics slots per group in the workspace
  LayerSrh srh;            // single-layer calls
};

int env_int(const char *name, int dflt) {
  const char *s = std::getenv(name);
  if (!s || !*s) return dflt;
  return std::atoi(s);
}

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
  for (int i = 0; i < 4; ++i) {
    if (strides[i] < 1) return fail(CKV_INVALID_ARGUMENT, "K/V strides must be >= 1");
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
  pl.rt_max = nmax * pl.th;
  if (pl.rt_max > 12)
    return fail(CKV_UNSUPPORTED,
                "ceil(window/16) * SRHs per group must be <= 12 (window %d, %d SRHs)", p->window,
                nmax);
  pl.head_end_mask = 0;
  for (int rt = 0; rt < 32; ++rt)
    if ((rt + 1) % pl.th == 0) pl.head_end_mask |= 1u << rt;
  return CKV_OK;
}

int check_mask(const ckv_problem *p, const uint8_t *mask, Plan &pl) {
  int st;
  if ((st = layer_srh(p, mask, 0, pl.srh))) return st;
  return set_row_tiles(p, pl.srh.nmax, pl);
}

// Units of the single-pass kernel in a sequence of L keys.
int fused_units(int L) { return (L + ckv::fused_unit_keys() - 1) / ckv::fused_unit_keys(); }

// The two-kernel path is the default.  CKV_PATH=single selects the
// single-pass kernel where it applies: every group's units must fit in half of
// the workgroups that can be resident at once (its progress condition is that
// one group per concurrently running launch fits; the margin covers two
// launches on different streams) and the batch must fit its ticket table.
void choose_path(const ckv_problem *p, Plan &pl) {
  pl.fused = false;
  const char *path = std::getenv("CKV_PATH");
  if (!path || std::string(path) != "single") return;
  if (p->index_mode == CKV_INDEX_LAYER) return;   // its groups may have no SRH
  if (p->batch > ckv::kFusedMaxBatch || p->dtype != CKV_BF16) return;
  const int resident = ckv::fused_resident_workgroups(1, p->head_dim, pl.rt_max);
  if (resident <= 0) return;
  int nmax = 0;
  for (int b = 0; b < p->batch; ++b)
    nmax = std::max(nmax, fused_units(p->cu_seqlens_host[b + 1] - p->cu_seqlens_host[b]));
  if (2 * nmax <= resident) {
    pl.fused = true;
    pl.n_units_max = nmax;
    pl.fused_grid = resident;
  }
}

// Chunk sizes of the two-kernel path: multiples of 512 keys (statistics: an
// even number of 2-tile groups for each of the 4 waves) and 992 + 32 halo keys
// (column sums: an even number of 2-tile groups for each of the 8 waves).
void set_chunks(const ckv_problem *p, Plan &pl) {
  pl.T = p->cu_seqlens_host[p->batch];
  pl.lmax = 0;
  for (int b = 0; b < p->batch; ++b)
    pl.lmax = std::max(pl.lmax, p->cu_seqlens_host[b + 1] - p->cu_seqlens_host[b]);
  int c1 = env_int("CKV_CHUNK1", 0), c2 = env_int("CKV_CHUNK2", 0);
  if (c1 <= 0 || c1 % 512 != 0) c1 = pick_chunk(p, 512, 4096, 256);
  if (c2 <= 0 || (c2 + 32) % 512 != 0 || c2 > ckv::kMaxChunk2) c2 = 992;   // even groups per chunk
  pl.chunk1 = c1;
  pl.chunk2 = c2;
  pl.max_chunks1 = std::max(1, (pl.lmax + c1 - 1) / c1);
  pl.max_chunks2 = std::max(1, (pl.lmax + c2 - 1) / c2);
}

// Workgroups of cpw chunks first, then at least `tail` chunks of every
// (sequence, group) one per workgroup, so the end of each scoring grid is made
// of short workgroups.
void set_lead(Plan &pl, int tail1, int tail2) {
  tail1 = env_int("CKV_TAIL1", tail1);
  tail2 = env_int("CKV_TAIL2", tail2);
  pl.lead1 = pl.cpw1 > 1 ? std::max(0, (pl.max_chunks1 - tail1) / pl.cpw1) : pl.max_chunks1;
  pl.lead2 = pl.cpw2 > 1 ? std::max(0, (pl.max_chunks2 - tail2) / pl.cpw2) : pl.max_chunks2;
}

// The block the single-pass kernel zeroes before it runs, from `start`:
// [0] ticket, [1] fallbacks, [64 ..) arrivals per (layer, group), then the
// published (normaliser, marker) pairs per (layer, group, row slot), then the
// first-digit histograms per (layer, group) (also used by the two-pass path).
void set_counters(const ckv_problem *p, Plan &pl, size_t start, int n_layers) {
  const size_t lg = (size_t)p->batch * p->n_kv_heads * n_layers;
  pl.counters_off = start;
  pl.bias_off = start + round_up((64 + lg) * sizeof(int), 256);
  pl.hist_off = pl.bias_off + round_up(lg * pl.rt_max * 16 * sizeof(float2), 256);
  pl.n_counters = (int)((pl.hist_off - pl.counters_off) / sizeof(int) + lg * ckv::kHistBins);
  pl.total = pl.hist_off + round_up(lg * ckv::kHistBins * sizeof(int), 256);
}

// Partial-statistics slots per group: enough for either path's chunking.
int partial_slots(const Plan &pl) {
  int parts = pl.max_chunks1;
  parts = std::max(parts, fused_units(pl.lmax));
  return parts;
}

// Single-layer workspace: a one-entry layer table (for the single-pass
// kernel), scores, partial row statistics, then the counters block.
void make_plan(const ckv_problem *p, Plan &pl, bool decide_path) {
  set_chunks(p, pl);
  set_lead(pl, 0, 0);
  pl.n_layers = 1;
  if (decide_path) choose_path(p, pl);
  pl.max_parts = partial_slots(pl);
  const size_t groups = (size_t)p->batch * p->n_kv_heads;
  pl.table_off = 0;
  pl.scores_off = round_up(sizeof(ckv::LayerDesc), 256);
  pl.stats_off =
      pl.scores_off + round_up((size_t)p->n_kv_heads * pl.T * sizeof(float), 256);
  set_counters(p, pl,
               pl.stats_off +
                   round_up(groups * pl.max_parts * (size_t)pl.rt_max * 16 * sizeof(float2), 256),
               1);
  pl.stats_layer = 0;
  pl.hist_layer = 0;
}

// One-chunk workgroups at the end of the multi-layer scoring grids, per
// (sequence, group) and layer.
constexpr int kTail1 = 4, kTail2 = 4;

// Multi-layer workspace: the layer table, then per layer the scores and the
// partial row statistics, then the counters block (per layer inside).
void make_plan_layers(const ckv_problem *p, int n_layers, Plan &pl, bool decide_path) {
  set_chunks(p, pl);
  pl.n_layers = n_layers;
  // Longer workgroups once there are enough of them: a few rounds of the
  // resident workgroups keep the tail short, and every round keeps its key
  // stream going across chunk boundaries.
  const int64_t units1 = (int64_t)p->batch * p->n_kv_heads * n_layers * pl.max_chunks1;
  const int64_t units2 = (int64_t)p->batch * p->n_kv_heads * n_layers * pl.max_chunks2;
  pl.cpw1 = (int)std::max<int64_t>(1, std::min<int64_t>(8, units1 / 3072));
  pl.cpw2 = (int)std::max<int64_t>(1, std::min<int64_t>(8, units2 / 2048));
  const int e1 = env_int("CKV_CPW1", 0), e2 = env_int("CKV_CPW2", 0);
  if (e1 > 0) pl.cpw1 = std::min(e1, 64);
  if (e2 > 0) pl.cpw2 = std::min(e2, 64);
  set_lead(pl, kTail1, kTail2);
  pl.fused = false;
  if (decide_path) choose_path(p, pl);
  pl.max_parts = partial_slots(pl);
  const size_t groups = (size_t)p->batch * p->n_kv_heads;
  pl.stats_layer = (int64_t)(groups * pl.max_parts * (size_t)pl.rt_max * 16);
  pl.hist_layer = (int64_t)(groups * ckv::kHistBins);
  pl.table_off = 0;
  pl.scores_off = round_up((size_t)n_layers * sizeof(ckv::LayerDesc), 256);
  pl.stats_off = pl.scores_off +
                 round_up((size_t)n_layers * p->n_kv_heads * pl.T * sizeof(float), 256);
  set_counters(p, pl,
               pl.stats_off + round_up((size_t)n_layers * pl.stats_layer * sizeof(float2), 256),
               n_layers);
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
  a.row_slots = pl.rt_max * 16;
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

ckv::SelectArgs select_args(const ckv_problem *p, const Plan &pl, const int *hist) {
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
  if (bits) bits->assign((size_t)n_layers * (ckv::kMaxQHeads / 32), 0u);
  for (int l = 0; l < n_layers; ++l) {
    const uint8_t *m = masks + (size_t)l * p->n_q_heads;
    if ((st = layer_srh(p, m, l, ls))) return st;
    nmax = std::max(nmax, ls.nmax);
    if (bits)
      for (int h = 0; h < p->n_q_heads; ++h)
        if (m[h]) (*bits)[(size_t)l * (ckv::kMaxQHeads / 32) + h / 32] |= 1u << (h % 32);
  }
  if ((st = set_row_tiles(p, nmax, pl))) return st;
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

// Enqueue the table writes of a multi-layer call.
hipError_t put_layers(const ckv_problem *p, const Plan &pl, int n_layers, const LayerPtrs &lp,
                      const std::vector<uint32_t> &bits, float *scores, void *ws,
                      hipStream_t stream) {
  ckv::LayerDesc *table =
      reinterpret_cast<ckv::LayerDesc *>(static_cast<char *>(ws) + pl.table_off);
  const size_t per_layer_scores = (size_t)p->n_kv_heads * pl.T;
  for (int first = 0; first < n_layers; first += ckv::kPutLayers) {
    ckv::PutArgs a{};
    a.table = table;
    a.first = first;
    a.count = std::min(ckv::kPutLayers, n_layers - first);
    a.Hq = p->n_q_heads;
    a.Hkv = p->n_kv_heads;
    for (int i = 0; i < a.count; ++i) {
      const int l = first + i;
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

// The single-pass kernel over n_layers layers of the table a.layers.
hipError_t launch_fused(const ckv_problem *p, const Plan &pl, const ckv::ScoreArgs &a, void *ws,
                        int n_layers, hipStream_t stream) {
  ckv::FusedArgs f{};
  f.s = a;
  int *ctr = reinterpret_cast<int *>(static_cast<char *>(ws) + pl.counters_off);
  f.ticket = ctr;
  f.fallbacks = ctr + 1;
  f.arrive = ctr + 64;
  f.bias = reinterpret_cast<float2 *>(static_cast<char *>(ws) + pl.bias_off);
  int acc = 0;
  for (int b = 0; b <= p->batch; ++b) {
    f.seq_units[b] = acc;
    if (b < p->batch)
      acc += p->n_kv_heads * fused_units(p->cu_seqlens_host[b + 1] - p->cu_seqlens_host[b]);
  }
  f.units_per_layer = acc;
  f.n_units_total = acc * n_layers;
  const int grid = std::min(pl.fused_grid, f.n_units_total);
  return ckv::launch_fused_score(f, p->dtype == CKV_BF16, p->head_dim, pl.rt_max, pl.n_counters,
                                 grid, stream);
}

// S1-S4 of a single-layer call on the path the plan chose.
hipError_t launch_scoring(const ckv_problem *p, const Plan &pl, const void *q, const void *k,
                          float *scores, void *ws, hipStream_t stream) {
  ckv::ScoreArgs a = score_args(p, pl, ws);
  a.l0 = layer_desc(&pl.srh, q, k, nullptr, scores, nullptr, nullptr, nullptr, 0);
  if (!pl.fused)
    return ckv::launch_score(a, p->dtype == CKV_BF16, p->head_dim, pl.rt_max, p->batch, stream);
  // the single-pass kernel reads its operands from a layer table
  LayerPtrs lp;
  lp.q = &q;
  lp.k = &k;
  std::vector<uint32_t> bits(ckv::kMaxQHeads / 32, 0u);
  for (uint8_t h : pl.srh.head) bits[h / 32] |= 1u << (h % 32);
  hipError_t e = put_layers(p, pl, 1, lp, bits, scores, ws, stream);
  if (e != hipSuccess) return e;
  a.layers = reinterpret_cast<const ckv::LayerDesc *>(static_cast<char *>(ws) + pl.table_off);
  return launch_fused(p, pl, a, ws, 1, stream);
}

// S1-S4 of a multi-layer call on the path the plan chose.
hipError_t launch_scoring_layers(const ckv_problem *p, const Plan &pl, const ckv::ScoreArgs &a,
                                 void *ws, int n_layers, hipStream_t stream) {
  if (!pl.fused)
    return ckv::launch_score_layers(a, p->dtype == CKV_BF16, p->head_dim, pl.rt_max, p->batch,
                                    n_layers, stream);
  return launch_fused(p, pl, a, ws, n_layers, stream);
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
  make_plan_layers(p, n_layers, pl, false);
  if ((st = check_ws(pl, ws, ws_bytes))) return st;
  make_plan_layers(p, n_layers, pl, true);
  float *scores = scores_or_null
                      ? scores_or_null
                      : reinterpret_cast<float *>(static_cast<char *>(ws) + pl.scores_off);
  hipStream_t s = (hipStream_t)stream;
  if ((st = hip_status(put_layers(p, pl, n_layers, lp, bits, scores, ws, s), "layer table")))
    return st;
  const ckv::LayerDesc *table =
      reinterpret_cast<const ckv::LayerDesc *>(static_cast<char *>(ws) + pl.table_off);
  ckv::ScoreArgs a = score_args(p, pl, ws);
  a.layers = table;
  if ((st = hip_status(launch_scoring_layers(p, pl, a, ws, n_layers, s), "score"))) return st;
  if ((st = hip_status(launch_combine_if_shared(p, pl, nullptr, nullptr, table, n_layers, s),
                       "combine")))
    return st;
  if (!full) return ok();
  ckv::SelectArgs sa = select_args(p, pl, a.hist);
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
  make_plan(p, pl, true);
  ok();
  return pl.fused ? 1 : 2;
}

size_t compresskv_workspace_bytes(const ckv_problem *p, const uint8_t *srh_mask_host,
                                  int32_t budget) {
  Plan pl;
  if (check_problem(p) || check_mask(p, srh_mask_host, pl) || check_budget(p, budget)) return 0;
  make_plan(p, pl, false);
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
  make_plan(p, pl, false);
  if ((st = check_ws(pl, ws, ws_bytes))) return st;
  make_plan(p, pl, true);
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
  ckv::SelectArgs sa = select_args(p, pl, nullptr);
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
  make_plan(p, pl, false);
  if ((st = check_ws(pl, ws, ws_bytes))) return st;
  make_plan(p, pl, true);
  float *scores = scores_or_null
                      ? scores_or_null
                      : reinterpret_cast<float *>(static_cast<char *>(ws) + pl.scores_off);
  hipStream_t s = (hipStream_t)stream;
  if ((st = hip_status(launch_scoring(p, pl, q_win, k, scores, ws, s), "score"))) return st;
  if ((st = hip_status(launch_combine_if_shared(p, pl, &pl.srh, scores, nullptr, 0, s),
                       "combine")))
    return st;
  const int *hist = reinterpret_cast<const int *>(static_cast<char *>(ws) + pl.hist_off);
  ckv::SelectArgs sa = select_args(p, pl, hist);
  sa.l0 = layer_desc(nullptr, nullptr, nullptr, nullptr, scores, idx, nullptr, nullptr, budget);
  if ((st = hip_status(ckv::launch_select(sa, 0, s), "select"))) return st;
  ckv::GatherArgs ga = gather_args(p);
  ga.l0 = layer_desc(nullptr, nullptr, k, v, nullptr, idx, k_out, v_out, budget);
  if ((st = hip_status(ckv::launch_gather(ga, 0, budget, s), "gather"))) return st;
  return ok();
}

size_t compresskv_layers_workspace_bytes(const ckv_problem *p, int32_t n_layers,
                                         const uint8_t *srh_masks_host) {
  Plan pl;
  if (check_problem(p) || check_layers(p, n_layers, srh_masks_host, LayerPtrs{}, pl, nullptr))
    return 0;
  make_plan_layers(p, n_layers, pl, false);
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
  ckv::SelectArgs sa = select_args(p, pl, nullptr);
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
  make_plan(p, pl, false);
  if ((st = check_ws(pl, ws, ws_bytes))) return st;
  make_plan(p, pl, true);
  float *scores = scores_or_null
                      ? scores_or_null
                      : reinterpret_cast<float *>(static_cast<char *>(ws) + pl.scores_off);
  hipStream_t s = (hipStream_t)stream;
  if ((st = hip_status(launch_scoring(p, pl, q_win, k, scores, ws, s), "score"))) return st;
  const int *hist = reinterpret_cast<const int *>(static_cast<char *>(ws) + pl.hist_off);
  ckv::SelectArgs sa = select_args(p, pl, hist);
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
