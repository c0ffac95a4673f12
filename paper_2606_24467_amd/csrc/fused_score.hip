// Single-pass scoring kernel (steps S1-S4) for gfx950.
//
// The window softmax (section 3.3, SnapKV-style window of section 4) needs a
// row's statistics over all keys of the sequence before any column sum can be
// formed.  The two-kernel path therefore streams K twice.  This kernel reads
// each key once: a workgroup holds a unit of one group's keys in registers,
// publishes the unit's partial row statistics, and forms the unit's window
// sums, pooled scores and selection histogram once every unit of the same
// (layer, sequence, KV group) has published and the last of them has merged
// the partials into the row normalisers.
//
// Persistent pipeline.  The grid is sized to the workgroups that can be
// resident; each workgroup loops, taking unit numbers from an atomic ticket.
// It holds two units: A (statistics published, column sums pending) and B
// (the next unit).  Per iteration it polls A's normalisers, issues B's loads,
// computes and publishes B's statistics, then finishes A (normally without
// waiting: A was published an iteration earlier).  Publishing never waits for
// another group, so groups complete as fast as their units are loaded.  Units
// are numbered layer by layer and group by group, so the units of a group are
// taken close together in time.
//
// Progress.  A workgroup blocks only on A's group, and only after publishing
// everything it holds; the last unit of a group to arrive merges the group
// before its workgroup does anything else.  Every blocking wait is therefore
// on a group whose units are all taken and published, or held by running
// workgroups that publish them without waiting, as long as the running
// workgroups number at least half the units of a group; the host requires
// twice that margin.  Every wait is bounded anyway: a wait that hits its bound
// is counted in the workspace and that unit's scores are then not valid.
//
// Normalisers.  The merger publishes each row's normaliser together with a
// marker in one 8-byte store; the waiting workgroups poll the pairs of their
// own rows.  Counters, published normalisers and histograms are zeroed by
// fill_kernel, launched just before on the same stream.
#include "score_common.h"

namespace ckv {

constexpr int kFusedWaves = 4;     // waves per workgroup
// Query fragments of up to 4 row tiles are kept in registers (as in the
// two-pass kernels); with two units of keys resident this allows one
// workgroup per CU.
constexpr bool kFusedQReg = true;

__global__ __launch_bounds__(256) void fill_kernel(int *p, int n) {
  for (int i = blockIdx.x * 256 + threadIdx.x; i < n; i += gridDim.x * 256) p[i] = 0;
}

// A unit: kUnitKeys consecutive keys of one (layer, sequence, KV group).
// Workgroup-uniform.
struct FUnit {
  int valid;
  int layer, b, g, u, n_u, s0, L, P, u0;
  int gi;     // b * Hkv + g
  int gl;     // layer * batch * Hkv + gi: index of the group's counters
  int nh, rt_n;
  LayerView lv;
};

template <int kUnitKeys>
__device__ __forceinline__ FUnit decode_unit(const FusedArgs &f, int ticket_any) {
  const ScoreArgs &a = f.s;
  // the ticket is workgroup-uniform: keep the whole decode in scalar registers
  const int ticket = __builtin_amdgcn_readfirstlane(ticket_any);
  FUnit x;
  x.valid = ticket < f.n_units_total;
  // an invalid ticket decodes to the last unit, so that every load it issues
  // stays in bounds (that unit is then neither published nor scored)
  const int tk = x.valid ? ticket : f.n_units_total - 1;
  x.layer = tk / f.units_per_layer;
  const int t = tk - x.layer * f.units_per_layer;
  int b = 0;
  while (b + 1 < a.batch && f.seq_units[b + 1] <= t) ++b;
  x.b = b;
  const cptr<int32_t> cu = to_const(a.cu);
  x.s0 = cu[b];
  x.L = cu[b + 1] - x.s0;
  x.n_u = (x.L + kUnitKeys - 1) / kUnitKeys;
  x.g = (t - f.seq_units[b]) / x.n_u;
  x.u = (t - f.seq_units[b]) - x.g * x.n_u;
  x.P = x.L - a.W;
  x.u0 = x.u * kUnitKeys;
  x.gi = b * a.Hkv + x.g;
  x.gl = x.layer * a.batch * a.Hkv + x.gi;
  x.lv = layer_view<true>(a, x.layer, x.g);
  x.nh = x.lv.nsrh;
  x.rt_n = x.nh * a.th;
  return x;
}

// The global loads of a unit: its queries (staged through registers) and its
// keys (tile w + NW*i of wave w).  Key indices are clamped into the sequence,
// so the key loads are unconditional.
template <typename T, int D, int RTM, int UT>
__device__ __forceinline__ void unit_loads(const ScoreArgs &a, const FUnit &x,
                                           uint4 (&qv)[QStage<T, D, RTM, 64 * kFusedWaves>::n],
                                           uint4 (&kf)[UT][Slices<T, D>::n]) {
  constexpr int NW = kFusedWaves, kUnitKeys = 16 * NW * UT;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int c = lane & 15, quad = lane >> 4;
  q_load<T, D, RTM, 64 * NW>(a, x.lv, x.b, x.rt_n, qv);
  const int k_last = min(x.L, x.u0 + kUnitKeys) - 1;
#pragma unroll
  for (int i = 0; i < UT; ++i)
    load_k_row<T, D>(a, x.lv.k, x.s0, min(x.u0 + 16 * (wave + NW * i) + c, k_last), x.g, quad,
                     kf[i]);
}

// The pooling halo of a unit: one key tile per wave (wave 0: the tile before
// the unit, the others: the tile after it; only waves 0 and 1 use theirs),
// loaded when the unit is finished.
template <typename T, int D, int UT>
__device__ __forceinline__ void halo_loads(const ScoreArgs &a, const FUnit &x,
                                           uint4 (&kh)[Slices<T, D>::n]) {
  constexpr int kUnitKeys = 16 * kFusedWaves * UT;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int c = lane & 15, quad = lane >> 4;
  const int hb = (wave == 0) ? x.u0 - 16 : x.u0 + kUnitKeys;
  load_k_row<T, D>(a, x.lv.k, x.s0, min(max(hb + c, 0), x.L - 1), x.g, quad, kh);
}

// Partial (ref, sum) statistics of every row over the unit's keys, merged over
// the quads and waves; thread r < rt_n*16 returns row r's pair.
template <typename T, int D, int RT, int UT>
__device__ __forceinline__ float2 unit_stats(const ScoreArgs &a, const FUnit &x,
                                             const uint4 (&kf)[UT][Slices<T, D>::n],
                                             const uint4 *q_lds, float2 (*part)[12 * 16]) {
  constexpr int NW = kFusedWaves, NS = Slices<T, D>::n, RQ = RegTiles<T, D, RT, kFusedQReg>::v;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int c = lane & 15, quad = lane >> 4;
  uint4 qreg[RegTiles<T, D, RT, kFusedQReg>::n][NS];
#pragma unroll
  for (int rt = 0; rt < RQ; ++rt)
#pragma unroll
    for (int s = 0; s < NS; ++s) qreg[rt][s] = q_frag<T, D>(q_lds, rt, s, c, quad);
  float ref[RT], sum[RT];
  bool ready = false;
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    ref[rt] = -INFINITY;
    sum[rt] = 0.f;
  }
#pragma unroll
  for (int i = 0; i < UT; ++i) {
    f32x4 acc[RT];
    tile_logits_all<T, D, RT, true, kFusedQReg>(kf[i], qreg, q_lds, c, quad, acc);
    stats_update<RT>(a, acc, ref, sum, ready, x.u0 + 16 * (wave + NW * i), x.L, x.P, c, quad);
  }
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
#pragma unroll
    for (int o = 16; o <= 32; o <<= 1) {
      const float ro = __shfl_xor(ref[rt], o);
      const float so = __shfl_xor(sum[rt], o);
      merge_stats(ref[rt], sum[rt], ro, so);
    }
  }
  if (quad == 0) {
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) part[wave][rt * 16 + c] = make_float2(ref[rt], sum[rt]);
  }
  __syncthreads();
  const int tid = threadIdx.x;
  float2 res = make_float2(-INFINITY, 0.f);
  if (tid < x.rt_n * 16) {
    float r0 = part[0][tid].x, s0 = part[0][tid].y;
#pragma unroll
    for (int w = 1; w < NW; ++w) merge_stats(r0, s0, part[w][tid].x, part[w][tid].y);
    res = make_float2(r0, s0);
  }
  __syncthreads();   // part is reused
  return res;
}

// Window sums of the unit's tiles and of its halo tiles into cs (cs[h][16 + x]
// = SRH h's window sum at key u0 + x, x = -16 .. kUnitKeys + 15).
template <typename T, int D, int RT, int UT, int CSW>
__device__ __forceinline__ void unit_window_sums(const ScoreArgs &a, const FUnit &x,
                                                 const uint4 (&kf)[UT][Slices<T, D>::n],
                                                 const uint4 (&kh)[Slices<T, D>::n],
                                                 const uint4 *q_lds, const float *bias_s,
                                                 float (*cs)[CSW]) {
  constexpr int NW = kFusedWaves, NS = Slices<T, D>::n, RQ = RegTiles<T, D, RT, kFusedQReg>::v;
  constexpr int kUnitKeys = 16 * NW * UT;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int c = lane & 15, quad = lane >> 4;
  uint4 qreg[RegTiles<T, D, RT, kFusedQReg>::n][NS];
#pragma unroll
  for (int rt = 0; rt < RQ; ++rt)
#pragma unroll
    for (int s = 0; s < NS; ++s) qreg[rt][s] = q_frag<T, D>(q_lds, rt, s, c, quad);
  float bias[RT][4];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int r = 0; r < 4; ++r) bias[rt][r] = bias_s[rt * 16 + 4 * quad + r];
#pragma unroll
  for (int i = 0; i < UT; ++i) {
    const int e = wave + NW * i;
    tile_window_sums<T, D, RT, CSW, kFusedQReg>(a, kf[i], qreg, q_lds, bias, e, x.u0 + 16 * e < x.P, c, quad,
                                    cs);
  }
  if (wave < 2) {
    const int hb = (wave == 0) ? x.u0 - 16 : x.u0 + kUnitKeys;
    tile_window_sums<T, D, RT, CSW, kFusedQReg>(a, kh, qreg, q_lds, bias, (wave == 0) ? -1 : kUnitKeys / 16,
                                    hb >= 0 && hb < x.P, c, quad, cs);
  }
}

// Grid: at most the resident workgroups, 64*kFusedWaves threads each; see the
// header for the pipeline.  Operands come from the layer table (a single-layer
// call uses a table of one layer).
template <typename T, int D, int RTM, int UT>
__global__ __launch_bounds__(64 * kFusedWaves) void fused_score_kernel(const FusedArgs f) {
  constexpr int NW = kFusedWaves, NT = 64 * NW, NS = Slices<T, D>::n;
  constexpr int kUnitKeys = 16 * NW * UT;
  constexpr int CSW = kUnitKeys + 32;
  constexpr int QN = QStage<T, D, RTM, NT>::n;
  constexpr int QSZ = RTM * 16 * QLayout<T, D>::STRIDE;
  const ScoreArgs &a = f.s;
  const int tid = threadIdx.x;

  __shared__ int tk_s, flag_s;
  __shared__ uint4 q_lds[2][QSZ];
  __shared__ float2 part[NW][12 * 16];
  __shared__ float bias_s[RTM * 16];
  __shared__ float cs[RTM][CSW];
  __shared__ float stage[kUnitKeys];
  __shared__ int hist_s[kHistBins];

  uint4 qv[QN];
  uint4 kf0[UT][NS], kf1[UT][NS], kh[NS];
  int pend_tk = 0;   // thread 0: the ticket taken for the next unit

  // Statistics of unit x (keys kf, queries staged in qv) via q_lds[qb] into
  // the published partials; returns true (uniformly) if x was the last unit of
  // its group to arrive, in which case the group's normalisers have been
  // merged into bias_s and published.
  auto publish = [&](const FUnit &x, const uint4 (&kf)[UT][NS],
                     int qb) __attribute__((always_inline)) -> bool {
    q_store<T, D, RTM, NT>(qv, q_lds[qb]);
    __syncthreads();
    float2 mine = make_float2(-INFINITY, 0.f);
    dispatch_rt<RTM>(x.rt_n, [&]<int RT>() {
      mine = unit_stats<T, D, RT, UT>(a, x, kf, q_lds[qb], part);
    });
    float2 *gparts = a.stats + x.layer * a.stats_layer +
                     ((int64_t)x.gi * a.parts_stride + x.u) * a.row_slots;
    if (tid < x.rt_n * 16) store_partial_coherent(gparts + tid, mine);
    // the partials (and every earlier store) reach the coherence point before
    // the arrival is counted
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    if (tid == 0) {
      const int before =
          __hip_atomic_fetch_add(&f.arrive[x.gl], 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      flag_s = (before == x.n_u - 1);
    }
    __syncthreads();
    if (!__builtin_amdgcn_readfirstlane(flag_s)) return false;
    // Last unit of the group: every partial is published.  Merge them (S2)
    // and publish the normalisers with their marker.
    const int rows = x.rt_n * 16;
    merge_row_bias<NT, true, 8>(a,
                             a.stats + x.layer * a.stats_layer +
                                 (int64_t)x.gi * a.parts_stride * a.row_slots,
                             a.row_slots, x.n_u, rows, RTM * 16, bias_s);
    __syncthreads();
    float2 *gbias = f.bias + (int64_t)x.gl * a.row_slots;
    if (tid < rows) store_partial_coherent(gbias + tid, make_float2(bias_s[tid], 1.f));
    return true;
  };

  // S3 + S4 of unit x once its group's normalisers are in bias_s.
  auto finish = [&](const FUnit &x, const uint4 (&kf)[UT][NS], const uint4 (&kh)[NS],
                    int qb) __attribute__((always_inline)) {
    dispatch_rt<RTM>(x.rt_n, [&]<int RT>() {
      unit_window_sums<T, D, RT, UT, CSW>(a, x, kf, kh, q_lds[qb], bias_s, cs);
    });
    for (int i = tid; i < kHistBins; i += NT) hist_s[i] = 0;
    const gptr<float> out = x.lv.scores + (int64_t)x.g * a.T + x.s0;
    // window positions of the unit are always kept: +inf
    for (int j = max(x.u0, x.P) + tid; j < min(x.L, x.u0 + kUnitKeys); j += NT) out[j] = INFINITY;
    __syncthreads();
    if (x.u0 < x.P) {
      pool_chunk<NT, CSW>(a, cs, x.nh, x.u0, min(x.u0 + kUnitKeys, x.P), x.P, out, stage,
                          hist_s);
      __syncthreads();
      flush_hist<NT>(hist_s, a.hist + x.layer * a.hist_layer + (int64_t)x.gi * kHistBins);
    }
    __syncthreads();   // cs, stage and hist_s are reused
  };

  // Normalisers of x's group into bias_s: the pairs polled before (pv, issued
  // ahead of the next unit's loads), polled again with a bounded wait until
  // every row carries the marker.
  auto await_bias = [&](const FUnit &x, float2 pv) __attribute__((always_inline)) {
    const int rows = x.rt_n * 16;
    const float2 *gbias = f.bias + (int64_t)x.gl * a.row_slots;
    int ok = __syncthreads_and(tid >= rows || pv.y == 1.f);
    int spins = 0;
    while (!ok) {
      __builtin_amdgcn_s_sleep(2);
      if (++spins > (1 << 16)) {
        if (tid == 0) atomicAdd(f.fallbacks, 1);
        break;
      }
      pv = load_partial_coherent(gbias + min(tid, rows - 1));
      ok = __syncthreads_and(tid >= rows || pv.y == 1.f);
    }
    if (tid < rows) bias_s[tid] = pv.x;
    for (int r = rows + tid; r < RTM * 16; r += NT) bias_s[r] = INFINITY;
    __syncthreads();
  };

  // One iteration with A in (kfa, q_lds[qa]); the next unit B goes to
  // (kfb, q_lds[1 - qa]).  Returns false when there is no next unit.
  auto iterate = [&](FUnit &A, int &qa, const uint4 (&kfa)[UT][NS],
                     uint4 (&kfb)[UT][NS]) __attribute__((always_inline)) -> bool {
    if (tid == 0) tk_s = pend_tk;
    __syncthreads();
    const FUnit B = decode_unit<kUnitKeys>(f, tk_s);
    __syncthreads();   // tk_s is written again before the next read
    if (tid == 0 && B.valid) pend_tk = atomicAdd(f.ticket, 1);
    // issue order = use order: A's normalisers, B's operands, A's halo
    const int rows_a = A.rt_n * 16;
    const float2 pv =
        load_partial_coherent(f.bias + (int64_t)A.gl * a.row_slots + min(tid, rows_a - 1));
    unit_loads<T, D, RTM, UT>(a, B, qv, kfb);
    halo_loads<T, D, UT>(a, A, kh);
    if (B.valid) publish(B, kfb, 1 - qa);
    await_bias(A, pv);
    finish(A, kfa, kh, qa);
    if (!B.valid) return false;
    A = B;
    qa = 1 - qa;
    return true;
  };

  // prologue: the first unit, published
  if (tid == 0) tk_s = atomicAdd(f.ticket, 1);
  __syncthreads();
  FUnit A = decode_unit<kUnitKeys>(f, tk_s);
  if (!A.valid) return;   // uniform
  if (tid == 0) pend_tk = atomicAdd(f.ticket, 1);
  unit_loads<T, D, RTM, UT>(a, A, qv, kf0);
  int qa = 0;
  publish(A, kf0, qa);
  for (;;) {
    if (!iterate(A, qa, kf0, kf1)) break;
    if (!iterate(A, qa, kf1, kf0)) break;
  }
}

// Built for bf16 keys with 256-key units and for 4, 6 or 12 row tiles (a
// group's tiles are rounded up to one of these, the extra ones holding zero
// queries).
constexpr int kFusedUnitTiles = 4;

__host__ __device__ constexpr int fused_rtm(int rt_max) {
  return rt_max <= 4 ? 4 : rt_max <= 6 ? 6 : 12;
}

static const void *fused_kernel_fn(int dtype_bf16, int head_dim, int rt_max) {
  if (!dtype_bf16 || rt_max > 12) return nullptr;
  constexpr int UT = kFusedUnitTiles;
  const int r = fused_rtm(rt_max);
  if (head_dim == 64)
    return r == 4   ? (const void *)fused_score_kernel<__bf16, 64, 4, UT>
           : r == 6 ? (const void *)fused_score_kernel<__bf16, 64, 6, UT>
                    : (const void *)fused_score_kernel<__bf16, 64, 12, UT>;
  return r == 4   ? (const void *)fused_score_kernel<__bf16, 128, 4, UT>
         : r == 6 ? (const void *)fused_score_kernel<__bf16, 128, 6, UT>
                  : (const void *)fused_score_kernel<__bf16, 128, 12, UT>;
}

int fused_unit_keys() { return 16 * kFusedWaves * kFusedUnitTiles; }

// Workgroups of the single-pass kernel that fit on the device at once (0: the
// configuration is not built, or the query failed).
int fused_resident_workgroups(int dtype_bf16, int head_dim, int rt_max) {
  const void *fn = fused_kernel_fn(dtype_bf16, head_dim, rt_max);
  if (!fn) return 0;
  int dev = 0, cus = 0, per_cu = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, 64 * kFusedWaves, 0) !=
      hipSuccess)
    return 0;
  return per_cu * cus;
}

// `counters` = number of ints from f.ticket on that fill_kernel zeroes
// (ticket, fallback count, arrivals, published normalisers and histograms,
// laid out contiguously by the host).  grid: persistent workgroups (at most
// the resident ones).
hipError_t launch_fused_score(const FusedArgs &f, int dtype_bf16, int head_dim, int rt_max,
                              int counters, int grid, hipStream_t stream) {
  const void *fn = fused_kernel_fn(dtype_bf16, head_dim, rt_max);
  if (!fn) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL(fill_kernel, dim3(256), dim3(256), 0, stream, f.ticket, counters);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  FusedArgs arg = f;
  void *params[] = {&arg};
  return hipLaunchKernel(fn, dim3(grid), dim3(64 * kFusedWaves), params, 0, stream);
}

}  // namespace ckv
