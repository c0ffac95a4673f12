// Single-pass scoring kernel (steps S1-S4) for gfx950.
//
// The window softmax (section 3.3, SnapKV-style window of section 4) needs a
// row's statistics over all keys of the sequence before any column sum can be
// formed.  The two-kernel path therefore streams K twice.  This kernel reads
// each key once: a workgroup loads one unit of a group's keys into registers,
// computes the unit's partial row statistics, publishes them, waits until
// every unit of the same (sequence, KV group) has published, merges the
// partials into the row normalisers and forms the window sums, pooled scores
// and selection histogram from the keys it still holds.
//
// Ordering and progress.  Units are numbered group by group (all units of
// group 0, then group 1, ...), and a workgroup takes the next number from an
// atomic ticket when it starts; the started workgroups always form a prefix of
// that numbering, so at most one group of a launch is waiting for units that
// have not started.  The last unit of a group to publish merges the partials
// and publishes the row normalisers; the others wait for that (never before
// publishing their own partials).  Hence the waits end whenever one group's
// units fit in the workgroups that can be resident at once, and, for k
// launches running concurrently, whenever k groups do; the host keeps a
// margin for two.  Every wait is bounded anyway: a wait that hits its bound
// is counted in the workspace and the unit's scores are then not valid.
//
// Two workgroups share a CU: while one waits for its group, the other
// streams keys.  Counters (ticket, per-group arrivals, histograms) are zeroed
// by fill_kernel, launched just before on the same stream.
#include "score_common.h"

namespace ckv {

constexpr int kFusedWaves = 4;     // waves per workgroup (two workgroups per CU)

__global__ __launch_bounds__(256) void fill_kernel(int *p, int n) {
  for (int i = blockIdx.x * 256 + threadIdx.x; i < n; i += gridDim.x * 256) p[i] = 0;
}

// Keys of a unit: tile w + NW*i (i < UT) of wave w, clamped into [.., k_last].
template <typename T, int D, int NW, int UT>
__device__ __forceinline__ void load_unit(const ScoreArgs &a, gptr<const char> kb, int s0, int g,
                                          int u0, int k_last, uint4 (&kf)[UT][Slices<T, D>::n]) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int c = lane & 15, quad = lane >> 4;
#pragma unroll
  for (int i = 0; i < UT; ++i)
    load_k_row<T, D>(a, kb, s0, min(u0 + 16 * (wave + NW * i) + c, k_last), g, quad, kf[i]);
}

// Partial (ref, sum) statistics of every row over the keys of one unit held in
// kf, merged over the quads and the waves; thread r < rt_n*16 returns row r's
// pair (others return an empty pair).
template <typename T, int D, int RTM, int NW, int UT>
__device__ __forceinline__ float2 unit_stats(const ScoreArgs &a,
                                             const uint4 (&kf)[UT][Slices<T, D>::n],
                                             const uint4 (&qreg)[RegTiles<T, D, RTM>::n]
                                                                [Slices<T, D>::n],
                                             const uint4 *q_lds, float2 (*part)[RTM * 16],
                                             int rt_n, int u0, int L, int P) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int c = lane & 15, quad = lane >> 4;
  float ref[RTM], sum[RTM];
  bool ready = false;
#pragma unroll
  for (int rt = 0; rt < RTM; ++rt) {
    ref[rt] = -INFINITY;
    sum[rt] = 0.f;
  }
#pragma unroll
  for (int i = 0; i < UT; ++i) {
    f32x4 acc[RTM];
#pragma unroll
    for (int rt = 0; rt < RTM; ++rt)
      acc[rt] = tile_logits<T, D, RTM, true>(kf[i], qreg, q_lds, rt, c, quad);
    stats_update<RTM>(a, acc, ref, sum, ready, u0 + 16 * (wave + NW * i), L, P, c, quad);
  }
#pragma unroll
  for (int rt = 0; rt < RTM; ++rt) {
#pragma unroll
    for (int o = 16; o <= 32; o <<= 1) {
      float ro = __shfl_xor(ref[rt], o);
      float so = __shfl_xor(sum[rt], o);
      merge_stats(ref[rt], sum[rt], ro, so);
    }
  }
  if (quad == 0) {
#pragma unroll
    for (int rt = 0; rt < RTM; ++rt) part[wave][rt * 16 + c] = make_float2(ref[rt], sum[rt]);
  }
  __syncthreads();
  const int tid = threadIdx.x;
  float2 res = make_float2(-INFINITY, 0.f);
  if (tid < rt_n * 16) {
    float r0 = part[0][tid].x, s_0 = part[0][tid].y;
#pragma unroll
    for (int w = 1; w < NW; ++w) merge_stats(r0, s_0, part[w][tid].x, part[w][tid].y);
    res = make_float2(r0, s_0);
  }
  __syncthreads();   // part is reused
  return res;
}

// Grid: n_units_total workgroups of 64*kFusedWaves threads.  A unit is
// 16 * kFusedWaves * UT keys of one (sequence, KV group).
template <typename T, int D, int RTM, int UT>
__global__ __launch_bounds__(64 * kFusedWaves) void fused_score_kernel(const FusedArgs f) {
  constexpr int NW = kFusedWaves;
  constexpr int NS = Slices<T, D>::n, RQ = RegTiles<T, D, RTM>::v;
  constexpr int NT = 64 * NW;
  constexpr int kUnitKeys = 16 * NW * UT;
  constexpr int CSW = kUnitKeys + 32;
  const ScoreArgs &a = f.s;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int c = lane & 15, quad = lane >> 4;

  __shared__ int ticket_s, waited_out, merger;
  __shared__ uint4 q_lds[RTM * 16 * QLayout<T, D>::STRIDE];
  __shared__ float2 part[NW][RTM * 16];
  __shared__ float bias_s[RTM * 16];
  __shared__ float cs[RTM][CSW];
  __shared__ int hist_s[kHistBins];

  if (tid == 0) ticket_s = atomicAdd(f.ticket, 1);
  __syncthreads();
  const int t = ticket_s;
  // ticket -> (sequence b, group g, unit u), group-major numbering
  int b = 0;
  while (b + 1 < a.batch && f.seq_units[b + 1] <= t) ++b;
  const int s0 = a.cu[b];
  const int L = a.cu[b + 1] - s0;
  const int n_u = (L + kUnitKeys - 1) / kUnitKeys;
  const int g = (t - f.seq_units[b]) / n_u;
  const int u = (t - f.seq_units[b]) - g * n_u;
  const int gi = b * a.Hkv + g;
  const int u0 = u * kUnitKeys;
  const int P = L - a.W;
  const LayerView lv = layer_view<false>(a, 0, g);
  const gptr<const char> kb = lv.k;
  const int nh = lv.nsrh;
  const int rt_n = nh * a.th;
  const int rows = rt_n * 16;

  // Loads: queries, the unit's keys, then the pooling halo tiles (wave 0: the
  // tile before the unit, wave 1: the tile after it).
  uint4 qv[QStage<T, D, RTM, NT>::n];
  q_load<T, D, RTM, NT>(a, lv, b, rt_n, qv);
  uint4 kf[UT][NS];
  load_unit<T, D, NW, UT>(a, kb, s0, g, u0, min(L, u0 + kUnitKeys) - 1, kf);
  const int halo_base = (wave == 0) ? u0 - 16 : u0 + kUnitKeys;
  const bool halo_ok = (wave < 2) && halo_base >= 0 && halo_base < P;
  uint4 kh[NS];
  if (wave < 2) load_k_row<T, D>(a, kb, s0, halo_ok ? min(halo_base + c, L - 1) : L - 1, g, quad, kh);
  q_store<T, D, RTM, NT>(qv, q_lds);
  for (int i = tid; i < kHistBins; i += NT) hist_s[i] = 0;
  __syncthreads();
  uint4 qreg[RegTiles<T, D, RTM>::n][NS];
#pragma unroll
  for (int rt = 0; rt < RQ; ++rt)
#pragma unroll
    for (int s = 0; s < NS; ++s) qreg[rt][s] = q_frag<T, D>(q_lds, rt, s, c, quad);

  // S1+S2: this unit's partial row statistics, published for the group.
  float2 *gparts = a.stats + (int64_t)gi * a.parts_stride * a.row_slots;
  const float2 mine = unit_stats<T, D, RTM, NW, UT>(a, kf, qreg, q_lds, part, rt_n, u0, L, P);
  if (tid < rows) store_partial_coherent(gparts + (int64_t)u * a.row_slots + tid, mine);
  // Every thread's partial store has reached the coherence point before the
  // arrival is counted (no cache-wide fence: the stores bypass the L2).
  __builtin_amdgcn_s_waitcnt(0);
  __syncthreads();
  // The group's normalisers live in the slot after its last partial.
  float2 *gbias = gparts + (int64_t)f.bias_slot * a.row_slots;
  if (tid == 0) {
    const int before =
        __hip_atomic_fetch_add(&f.arrive[gi], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    merger = (before == n_u - 1);
  }
  __syncthreads();
  if (merger) {
    // Last unit of the group: every partial is published.  Merge them (S2),
    // publish the row normalisers, then raise the group's ready flag.
    merge_row_bias<NT, true>(a, gparts, a.row_slots, n_u, rows, RTM * 16, bias_s);
    __syncthreads();
    if (tid < rows) store_partial_coherent(gbias + tid, make_float2(bias_s[tid], 0.f));
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (tid == 0)
      __hip_atomic_store(&f.ready[gi], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  } else {
    // Wait for the group's normalisers (bounded; see the header).
    if (tid == 0) {
      int spins = 0;
      waited_out = 0;
      while (__hip_atomic_load(&f.ready[gi], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0) {
        __builtin_amdgcn_s_sleep(4);
        if (++spins > (1 << 20)) {
          waited_out = 1;
          break;
        }
      }
    }
    __syncthreads();
    // A wait that hit its bound is counted (the unit's scores are then not
    // valid); with the host's group-size check it cannot happen unless more
    // single-pass kernels than that check allows run on the GPU at once.
    if (waited_out && tid == 0) atomicAdd(f.fallbacks, 1);
    if (tid < rows) bias_s[tid] = load_partial_coherent(gbias + tid).x;
    for (int r = rows + tid; r < RTM * 16; r += NT) bias_s[r] = INFINITY;
  }
  __syncthreads();
  float bias[RTM][4];
#pragma unroll
  for (int rt = 0; rt < RTM; ++rt)
#pragma unroll
    for (int r = 0; r < 4; ++r) bias[rt][r] = bias_s[rt * 16 + 4 * quad + r];

  // S3: window sums of the unit's tiles plus the halo tiles.
  // cs[h][16 + x] = window sum of SRH h at key u0 + x (x = -16 .. kUnitKeys + 15).
#pragma unroll
  for (int i = 0; i < UT; ++i) {
    const int e = wave + NW * i;
    tile_window_sums<T, D, RTM, CSW>(a, kf[i], qreg, q_lds, bias, e, u0 + 16 * e < P, c, quad,
                                     cs);
  }
  if (wave < 2)
    tile_window_sums<T, D, RTM, CSW>(a, kh, qreg, q_lds, bias, (wave == 0) ? -1 : kUnitKeys / 16,
                                     halo_ok, c, quad, cs);
  const gptr<float> out = lv.scores + (int64_t)g * a.T + s0;
  // Window positions of the unit are always kept: +inf.
  for (int j = max(u0, P) + tid; j < min(L, u0 + kUnitKeys); j += NT) out[j] = INFINITY;
  __syncthreads();
  // S4: pooling, SRH mean, histogram of the first selection digit.
  if (u0 < P) pool_scores<NT, CSW>(a, cs, nh, u0, min(u0 + kUnitKeys, P), P, out, hist_s);
  __syncthreads();
  flush_hist<NT>(hist_s, a.hist + (int64_t)gi * kHistBins);
}

template <typename T, int D, int RTM>
static hipError_t launch_fused_t(const FusedArgs &f, int unit_tiles, int counters,
                                 hipStream_t stream) {
  hipLaunchKernelGGL(fill_kernel, dim3(64), dim3(256), 0, stream, f.ticket, counters);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (unit_tiles == 2)
    hipLaunchKernelGGL((fused_score_kernel<T, D, RTM, 2>), dim3(f.n_units_total),
                       dim3(64 * kFusedWaves), 0, stream, f);
  else
    hipLaunchKernelGGL((fused_score_kernel<T, D, RTM, 4>), dim3(f.n_units_total),
                       dim3(64 * kFusedWaves), 0, stream, f);
  return hipGetLastError();
}

template <typename T, int D>
static hipError_t launch_fused_d(const FusedArgs &f, int rt_max, int unit_tiles, int counters,
                                 hipStream_t s) {
  switch (rt_max) {
    case 1: return launch_fused_t<T, D, 1>(f, unit_tiles, counters, s);
    case 2: return launch_fused_t<T, D, 2>(f, unit_tiles, counters, s);
    case 3: return launch_fused_t<T, D, 3>(f, unit_tiles, counters, s);
    case 4: return launch_fused_t<T, D, 4>(f, unit_tiles, counters, s);
    case 5:
    case 6: return launch_fused_t<T, D, 6>(f, unit_tiles, counters, s);
    case 7:
    case 8: return launch_fused_t<T, D, 8>(f, unit_tiles, counters, s);
    default: return launch_fused_t<T, D, 12>(f, unit_tiles, counters, s);
  }
}

// `counters` = number of ints from f.ticket on that fill_kernel zeroes (ticket,
// fallback count, arrivals and the histograms, laid out contiguously by the
// host).  unit_tiles: key tiles per wave per unit (2 or 4).
hipError_t launch_fused_score(const FusedArgs &f, int dtype_bf16, int head_dim, int rt_max,
                              int unit_tiles, int counters, hipStream_t stream) {
  if (dtype_bf16) {
    return head_dim == 64 ? launch_fused_d<__bf16, 64>(f, rt_max, unit_tiles, counters, stream)
                          : launch_fused_d<__bf16, 128>(f, rt_max, unit_tiles, counters, stream);
  }
  return head_dim == 64 ? launch_fused_d<float, 64>(f, rt_max, unit_tiles, counters, stream)
                        : launch_fused_d<float, 128>(f, rt_max, unit_tiles, counters, stream);
}

// Workgroups of one fused kernel that fit on the device at once (for the
// group-size check of the host).
int fused_resident_workgroups(int dtype_bf16, int head_dim, int rt_max, int unit_tiles) {
  int dev = 0, cus = 0, per_cu = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return 0;
  const void *fn = nullptr;
#define CKV_FN(T, D, R)                                                                  \
  fn = unit_tiles == 2 ? (const void *)fused_score_kernel<T, D, R, 2>                  \
                       : (const void *)fused_score_kernel<T, D, R, 4>
#define CKV_RT(T, D)                      \
  switch (rt_max) {                       \
    case 1: CKV_FN(T, D, 1); break;       \
    case 2: CKV_FN(T, D, 2); break;       \
    case 3: CKV_FN(T, D, 3); break;       \
    case 4: CKV_FN(T, D, 4); break;       \
    case 5: case 6: CKV_FN(T, D, 6); break; \
    case 7: case 8: CKV_FN(T, D, 8); break; \
    default: CKV_FN(T, D, 12); break;     \
  }
  if (dtype_bf16) {
    if (head_dim == 64) { CKV_RT(__bf16, 64) } else { CKV_RT(__bf16, 128) }
  } else {
    if (head_dim == 64) { CKV_RT(float, 64) } else { CKV_RT(float, 128) }
  }
#undef CKV_RT
#undef CKV_FN
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, 64 * kFusedWaves, 0) !=
      hipSuccess)
    return 0;
  return per_cu * cus;
}

}  // namespace ckv
