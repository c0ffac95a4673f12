// Device building blocks shared by the scoring kernels (steps S1-S4):
// query staging, key loads, MFMA tile logits, the running row statistics of
// the window softmax, the merge of row-statistics partials, and the pooling
// of window sums with the first-digit histogram of the selection.
//
// Rows of a KV group: SRH h (in head order) owns th = ceil(W/16) row tiles of
// 16 rows; row i < W of the tile set is window query i of that head, the
// padding rows have zero queries and are ignored.
#pragma once

#include "ckv_device.h"

namespace ckv {

template <typename T, int D>
struct QLayout {
  static constexpr int NS = Slices<T, D>::n;   // 16-byte slices per row and quad
  static constexpr int U4 = 4 * NS;            // 16-byte units per row
  static constexpr int STRIDE = U4 + 1;        // padded row stride in LDS (bank spread)
};

constexpr int kWaves = 4;       // waves per column-sum workgroup (two per CU: one streams
                                // keys while the other pools its chunk)
constexpr int kRing = 4;        // key tiles per wave in the load ring: kRing - 1 in flight
                                // while one is consumed

// Row tiles kept in registers: all of them when they fit in 64 VGPRs (and QR
// allows it), else none.
template <typename T, int D, int RTM, bool QR = true>
struct RegTiles {
  static constexpr int v = QR && RTM * Slices<T, D>::n <= 16 ? RTM : 0;
  static constexpr int n = v > 0 ? v : 1;   // array extent
};

// The group's SRH window queries (rt_n row tiles) staged in LDS in two
// phases: q_load issues every global load (before the first key loads, so that
// waiting for the queries never waits for keys), q_store writes them to LDS.
// Rows past W and tiles past rt_n are zero.
template <typename T, int D, int RTM, int NT>
struct QStage {
  static constexpr int U4 = QLayout<T, D>::U4;
  static constexpr int n = (RTM * 16 * U4 + NT - 1) / NT;   // 16-byte units per thread
};

template <typename T, int D, int RTM, int NT>
__device__ __forceinline__ void q_load(const ScoreArgs &a, const LayerView &lv, int b, int rt_n,
                                       uint4 (&qv)[QStage<T, D, RTM, NT>::n]) {
  constexpr int U4 = QLayout<T, D>::U4;
  const gptr<const char> qb = lv.q;
  // the group's SRH head indices, one per lane, read once: the query loads
  // then depend on a single load instead of one per row
  int hv = 0;
  if ((int)(threadIdx.x & 63) < lv.nsrh) hv = lv.srh_head[lv.off + (threadIdx.x & 63)];
#pragma unroll
  for (int it = 0; it < QStage<T, D, RTM, NT>::n; ++it) {
    const int idx = (int)threadIdx.x + it * NT;
    const int row = idx / U4, u = idx - row * U4;
    const int rt = row >> 4, c = row & 15;
    qv[it] = make_uint4(0, 0, 0, 0);
    const int head = __shfl(hv, min(rt / a.th, 63));   // every lane takes part
    if (rt < rt_n) {
      const int i = (rt % a.th) * 16 + c;
      if (i < a.W) {
        qv[it] = load16(qb + (((int64_t)b * a.W + i) * a.Hq + head) * (int64_t)(D * sizeof(T)) +
                        16 * u);
      }
    }
  }
}

template <typename T, int D, int RTM, int NT>
__device__ __forceinline__ void q_store(const uint4 (&qv)[QStage<T, D, RTM, NT>::n],
                                        uint4 *q_lds) {
  constexpr int U4 = QLayout<T, D>::U4, STRIDE = QLayout<T, D>::STRIDE;
#pragma unroll
  for (int it = 0; it < QStage<T, D, RTM, NT>::n; ++it) {
    const int idx = (int)threadIdx.x + it * NT;
    const int row = idx / U4, u = idx - row * U4;
    if (row < RTM * 16) q_lds[row * STRIDE + u] = qv[it];
  }
}

template <typename T, int D>
__device__ __forceinline__ uint4 q_frag(const uint4 *q_lds, int rt, int s, int c, int quad) {
  return q_lds[(rt * 16 + c) * QLayout<T, D>::STRIDE + 4 * s + quad];
}

// Slices of one key row of the layer's K at kb (key index clamped into the
// sequence by the callers).
template <typename T, int D>
__device__ __forceinline__ void load_k_row(const ScoreArgs &a, gptr<const char> kb, int s0,
                                           int key, int g, int quad,
                                           uint4 (&out)[Slices<T, D>::n]) {
  const gptr<const char> p = kb +
                  ((int64_t)(s0 + key) * a.k_stride_tok + (int64_t)g * a.k_stride_head) *
                      (int64_t)sizeof(T) +
                  16 * quad;
#pragma unroll
  for (int s = 0; s < Slices<T, D>::n; ++s) out[s] = load16(p + 64 * s);
}

// logits of row tile rt against one key tile; KEYS_AS_A selects the operand
// order (true: lane holds 4 keys of one row; false: 4 rows of one key).
template <typename T, int D, int RTM, bool KEYS_AS_A, bool QR = true>
__device__ __forceinline__ f32x4 tile_logits(const uint4 (&kf)[Slices<T, D>::n],
                                             const uint4 (&qreg)[RegTiles<T, D, RTM, QR>::n]
                                                                [Slices<T, D>::n],
                                             const uint4 *q_lds, int rt, int c, int quad) {
  constexpr int NS = Slices<T, D>::n, RQ = RegTiles<T, D, RTM, QR>::v;
  f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < NS; ++s) {
    uint4 qv;
    if (rt < RQ) {
      qv = qreg[rt < RQ ? rt : 0][s];   // rt < RQ here; the clamp only keeps the index static
    } else {
      qv = q_frag<T, D>(q_lds, rt, s, c, quad);
    }
    acc = KEYS_AS_A ? mfma_slice<T>(kf[s], qv, acc) : mfma_slice<T>(qv, kf[s], acc);
  }
  return acc;
}

// Logits of every row tile against one key tile, slice-major: the RT
// accumulation chains are independent, so the matrix pipeline interleaves
// them instead of waiting on one chain at a time.  Each tile accumulates its
// slices in the same order as tile_logits.
// SB (slice barrier): no instruction moves across the end of a slice, so only
// one slice's query fragments are read ahead from LDS at a time; kernels
// compiled for many row tiles use it to keep their register count at two
// waves per SIMD.
template <typename T, int D, int RT, bool KEYS_AS_A, bool QR = true, bool SB = false>
__device__ __forceinline__ void tile_logits_all(const uint4 (&kf)[Slices<T, D>::n],
                                                const uint4 (&qreg)[RegTiles<T, D, RT, QR>::n]
                                                                   [Slices<T, D>::n],
                                                const uint4 *q_lds, int c, int quad,
                                                f32x4 (&acc)[RT]) {
  constexpr int NS = Slices<T, D>::n, RQ = RegTiles<T, D, RT, QR>::v;
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) acc[rt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int s = 0; s < NS; ++s) {
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      uint4 qv;
      if (rt < RQ) {
        qv = qreg[rt < RQ ? rt : 0][s];
      } else {
        qv = q_frag<T, D>(q_lds, rt, s, c, quad);
      }
      acc[rt] = KEYS_AS_A ? mfma_slice<T>(kf[s], qv, acc[rt]) : mfma_slice<T>(qv, kf[s], acc[rt]);
    }
    if constexpr (SB && RQ < RT) __builtin_amdgcn_sched_barrier(0);
  }
}

// Row-tile counts the scoring loops are compiled for: a group with rt_n row
// tiles runs the smallest of them that is >= rt_n; the extra tiles hold zero
// queries (their rows are never read back), so every loop over row tiles has
// a compile-time bound and no branch.
__host__ __device__ constexpr int rt_class(int rt_n) {
  return rt_n <= 4 ? rt_n : rt_n <= 6 ? 6 : rt_n <= 8 ? 8 : rt_n <= 12 ? 12 : 16;
}

// Calls body.template operator()<RT>() with RT = rt_class(rt_n) (<= RTM).
template <int RTM, typename F>
__device__ __forceinline__ void dispatch_rt(int rt_n, F &&body) {
  switch (rt_class(rt_n)) {
    case 1: if constexpr (RTM >= 1) body.template operator()<1>(); break;
    case 2: if constexpr (RTM >= 2) body.template operator()<2>(); break;
    case 3: if constexpr (RTM >= 3) body.template operator()<3>(); break;
    case 4: if constexpr (RTM >= 4) body.template operator()<4>(); break;
    case 6: if constexpr (RTM >= 6) body.template operator()<6>(); break;
    case 8: if constexpr (RTM >= 8) body.template operator()<8>(); break;
    case 12: if constexpr (RTM >= 12) body.template operator()<12>(); break;
    default: if constexpr (RTM >= 16) body.template operator()<16>(); break;
  }
}

// Sum of v over the four quads (lanes c, c + 16, c + 32, c + 48) in every lane,
// with the gfx950 lane-swap instructions (no LDS round trip).
__device__ __forceinline__ float quad_sum(float v) {
  const auto s32 = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v),
                                                    false, false);
  v = __uint_as_float(s32[0]) + __uint_as_float(s32[1]);
  const auto s16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v),
                                                    false, false);
  return __uint_as_float(s16[0]) + __uint_as_float(s16[1]);
}

// Fold one key tile (logits acc[rt], keys base + 4*quad + r) into the running
// (ref, sum) pairs of this lane's rows, sum = sum_j exp2(y_j - ref).  A row's
// reference stays fixed while its sum stays below 2^64, so on the common path
// (every key of the tile is a prefix key and the references are set: `ready`)
// a logit costs one fma, one exp2 and one add.  The first tile, masked tiles
// (keys past the sequence end, or after the row's own position inside the
// window: causal) and a tile that would push a sum past 2^64 take the general
// path, which rebases a row on its largest new value when a term would exceed
// 2^30 (always the case for the first key of a row).
template <int RT>
__device__ __forceinline__ void stats_update(const ScoreArgs &a, const f32x4 (&acc)[RT],
                                             float (&ref)[RT], float (&sum)[RT], bool &ready,
                                             int base, int L, int P, int c, int quad) {
  constexpr float kRescale = 30.f;
  const bool unmasked = (base + 16 <= P);   // uniform
  if (ready && unmasked) {
    float s_new[RT];
    bool over = false;
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      // (e0 + e1) + e2 + e3: the terms are never -0, so this is 0 + e0 + ...
      float t = fast_exp2(__builtin_fmaf(acc[rt][0], a.c1, -ref[rt]));
#pragma unroll
      for (int r = 1; r < 4; ++r) t += fast_exp2(__builtin_fmaf(acc[rt][r], a.c1, -ref[rt]));
      s_new[rt] = sum[rt] + t;
      over |= !(s_new[rt] <= 0x1p64f);   // also true for inf and nan
    }
    if (!__any(over)) {
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) sum[rt] = s_new[rt];
      return;
    }
  }
  float d[RT][4];
  float dmax = -INFINITY;
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int i = (rt % a.th) * 16 + c;   // window index of this lane's row
      const int j = base + 4 * quad + r;
      const bool ok = unmasked || ((j < L) && (i >= a.W || j <= P + i));
      d[rt][r] = ok ? __builtin_fmaf(acc[rt][r], a.c1, -ref[rt]) : -INFINITY;
      dmax = fmaxf(dmax, d[rt][r]);
    }
  }
  if (__any(dmax > kRescale)) {
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      const float m = fmaxf(fmaxf(d[rt][0], d[rt][1]), fmaxf(d[rt][2], d[rt][3]));
      if (m > kRescale) {
        float best = -INFINITY;
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (d[rt][r] != -INFINITY) best = fmaxf(best, acc[rt][r] * a.c1);
        sum[rt] = (ref[rt] == -INFINITY) ? 0.f : sum[rt] * fast_exp2(ref[rt] - best);
        ref[rt] = best;
#pragma unroll
        for (int r = 0; r < 4; ++r)
          d[rt][r] = (d[rt][r] == -INFINITY) ? -INFINITY
                                             : __builtin_fmaf(acc[rt][r], a.c1, -best);
      }
    }
  }
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
#pragma unroll
    for (int r = 0; r < 4; ++r) sum[rt] += fast_exp2(d[rt][r]);
  }
  // after an unmasked tile every row has a finite reference
  ready = ready || unmasked;
}

// A partial (ref, sum) pair read or written at agent scope: the access goes to
// the device's coherence point instead of the per-XCD L2, so partials that
// workgroups of the same kernel exchange need no cache-wide fences.
__device__ __forceinline__ void store_partial_coherent(float2 *p, float2 v) {
  __hip_atomic_store(reinterpret_cast<unsigned long long *>(p),
                     __builtin_bit_cast(unsigned long long, v), __ATOMIC_RELAXED,
                     __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float2 load_partial_coherent(const float2 *p) {
  return __builtin_bit_cast(float2, __hip_atomic_load(
                                        reinterpret_cast<const unsigned long long *>(p),
                                        __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
}

// Row normalisers bias = ref + log2(sum) for the `rows` rows of one group,
// merged from n_parts partial (ref, sum) pairs laid out parts[k * stride + row]
// (fixed order per thread, then a shuffle tree over tpr threads per row).
// Padding rows (window index >= W) and rows >= rows get +inf.  COHERENT reads
// the partials at agent scope (they were written by this kernel).
template <int NT, bool COHERENT = false, int kBatch = 8>
__device__ __forceinline__ void merge_row_bias(const ScoreArgs &a, const float2 *parts,
                                               int64_t stride, int n_parts, int rows,
                                               int rows_cap, float *bias_s) {
  const int tid = threadIdx.x;
  int tpr = 1;
  while (tpr * 2 * rows <= NT && tpr < 32) tpr *= 2;
  const int row = tid / tpr, sub = tid % tpr;
  float m = -INFINITY, sm = 0.f;
  if (row < rows) {
    // batches of kBatch loads in flight, merged in index order
    for (int k0 = sub; k0 < n_parts; k0 += kBatch * tpr) {
      float2 v[kBatch];
#pragma unroll
      for (int j = 0; j < kBatch; ++j) {
        const int k = min(k0 + j * tpr, n_parts - 1);
        v[j] = COHERENT ? load_partial_coherent(parts + (int64_t)k * stride + row)
                        : parts[(int64_t)k * stride + row];
      }
#pragma unroll
      for (int j = 0; j < kBatch; ++j)
        if (k0 + j * tpr < n_parts) merge_stats(m, sm, v[j].x, v[j].y);
    }
  }
  for (int o = 1; o < tpr; o <<= 1) {
    const float mo = __shfl_xor(m, o), so = __shfl_xor(sm, o);
    merge_stats(m, sm, mo, so);
  }
  if (row < rows && sub == 0) {
    const int i = row % (16 * a.th);
    bias_s[row] = (i < a.W) ? m + fast_log2(sm) : INFINITY;
  }
  for (int r = rows + tid; r < rows_cap; r += NT) bias_s[r] = INFINITY;
}

// merge_row_bias over partials that other workgroups of the same launch
// publish: each is read at agent scope and carries its own arrival mark (the
// sum is stored negated, so a set sign bit means written; the slots start at
// +0 and a sum is never negative).  Until every partial has arrived the reads
// are repeated, at most `spin` more times; returns false (uniformly) if one
// never arrived.  Same merge order and arithmetic as merge_row_bias.
template <int NT, int kBatch = 8>
__device__ __forceinline__ bool merge_row_bias_marked(const ScoreArgs &a, const float2 *parts,
                                                      int64_t stride, int n_parts, int rows,
                                                      int rows_cap, float *bias_s, int spin) {
  const int tid = threadIdx.x;
  int tpr = 1;
  while (tpr * 2 * rows <= NT && tpr < 32) tpr *= 2;
  const int row = tid / tpr, sub = tid % tpr;
  float m, sm;
  for (int attempt = 0;; ++attempt) {
    m = -INFINITY;
    sm = 0.f;
    bool mine = true;
    if (row < rows) {
      for (int k0 = sub; k0 < n_parts; k0 += kBatch * tpr) {
        float2 v[kBatch];
#pragma unroll
        for (int j = 0; j < kBatch; ++j) {
          const int k = min(k0 + j * tpr, n_parts - 1);
          v[j] = load_partial_coherent(parts + (int64_t)k * stride + row);
        }
#pragma unroll
        for (int j = 0; j < kBatch; ++j) {
          if (k0 + j * tpr < n_parts) {
            mine = mine && signbit(v[j].y);
            merge_stats(m, sm, v[j].x, -v[j].y);
          }
        }
      }
    }
    if (__syncthreads_and(mine)) break;
    if (attempt >= spin) return false;
    __builtin_amdgcn_s_sleep(4);
  }
  for (int o = 1; o < tpr; o <<= 1) {
    const float mo = __shfl_xor(m, o), so = __shfl_xor(sm, o);
    merge_stats(m, sm, mo, so);
  }
  if (row < rows && sub == 0) {
    const int i = row % (16 * a.th);
    bias_s[row] = (i < a.W) ? m + fast_log2(sm) : INFINITY;
  }
  for (int r = rows + tid; r < rows_cap; r += NT) bias_s[r] = INFINITY;
  return true;
}

// Row normalisers that another workgroup of the same launch merged and
// published (rows_cap entries (bias, -1): the set sign bit marks them
// written, the slots start at +0), read at agent scope into bias_s; the reads
// are repeated at most `spin` more times; false (uniformly) if one never
// arrived.
template <int NT>
__device__ __forceinline__ bool read_bias_marked(const float2 *bias_g, int rows_cap,
                                                 float *bias_s, int spin) {
  const int tid = threadIdx.x;
  for (int attempt = 0;; ++attempt) {
    bool mine = true;
    for (int r = tid; r < rows_cap; r += NT) {
      const float2 v = load_partial_coherent(bias_g + r);
      mine = mine && signbit(v.y);
      bias_s[r] = v.x;
    }
    if (__syncthreads_and(mine)) return true;
    if (attempt >= spin) return false;
    __builtin_amdgcn_s_sleep(4);
  }
}

// Window sums of one key tile for every SRH of the group (MFMA operands: A =
// window rows, B = keys; lane (quad, c) holds rows 4*quad .. 4*quad+3 against
// key c): in-lane over the 4 rows and the SRH's row tiles, then across the
// quads.  cs[h][16 + 16*e + c] receives SRH h's sum for key c of tile e.  Row
// tiles past the group's own (zero queries) have bias +inf and add nothing.
// The VALU half of tile_window_sums: window sums of a tile from its logits.
template <int RT, int CSW>
__device__ __forceinline__ void window_sums_from_logits(const ScoreArgs &a, const f32x4 (&acc)[RT],
                                                        const float (&bias)[RT][4], int e,
                                                        bool keep, int c, int quad,
                                                        float (*cs)[CSW]) {
  // per row tile: the lane's 4 rows (no branch between the row tiles); the
  // terms are never -0, so starting from the first term equals starting from 0
  float vt[RT];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    vt[rt] = fast_exp2(__builtin_fmaf(acc[rt][0], a.c1, -bias[rt][0]));
#pragma unroll
    for (int r = 1; r < 4; ++r) vt[rt] += fast_exp2(__builtin_fmaf(acc[rt][r], a.c1, -bias[rt][r]));
  }
  // per SRH: its row tiles, then the quads
  int hh = 0;
  float v = 0.f;
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    v += vt[rt];
    if ((a.head_end_mask >> rt) & 1u) {
      v = quad_sum(v);
      if (keep && quad == (hh & 3)) cs[hh][16 + 16 * e + c] = v;
      v = 0.f;
      ++hh;
    }
  }
}

template <typename T, int D, int RT, int CSW, bool QR = true>
__device__ __forceinline__ void tile_window_sums(const ScoreArgs &a,
                                                 const uint4 (&kf)[Slices<T, D>::n],
                                                 const uint4 (&qreg)[RegTiles<T, D, RT, QR>::n]
                                                                    [Slices<T, D>::n],
                                                 const uint4 *q_lds, const float (&bias)[RT][4],
                                                 int e, bool keep, int c, int quad,
                                                 float (*cs)[CSW]) {
  f32x4 acc[RT];
  tile_logits_all<T, D, RT, false, QR>(kf, qreg, q_lds, c, quad, acc);
  window_sums_from_logits<RT, CSW>(a, acc, bias, e, keep, c, quad, cs);
}

// Pooling along the token axis (positions clipped to the prefix [0, P)), then
// the mean over the group's nh SRHs, for positions [c0, p_end); cs[h][16 + x]
// holds the window sum at key c0 + x (x from -16).  Each score goes to `out`
// and to the LDS histogram of its top 11 value bits.
template <int NT, int CSW>
__device__ __forceinline__ void pool_scores(const ScoreArgs &a, const float (*cs)[CSW],
                                            int nh, int c0, int p_end, int P, gptr<float> out,
                                            int *hist_s) {
  const int rp = (a.pool_kernel - 1) >> 1;
  const float inv_k = 1.f / (float)a.pool_kernel;
  const float inv_n = 1.f / (float)nh;
  for (int j = c0 + (int)threadIdx.x; j < p_end; j += NT) {
    const int lo = max(j - rp, 0) - c0 + 16;
    const int hi = min(j + rp, P - 1) - c0 + 16;
    float score;
    if (a.reduce_order == 0) {      // pool each SRH, then average
      score = 0.f;
      for (int h = 0; h < nh; ++h) {
        float v;
        if (a.pool_type == 0) {
          v = -INFINITY;
          for (int x = lo; x <= hi; ++x) v = fmaxf(v, cs[h][x]);
        } else {
          v = 0.f;
          for (int x = lo; x <= hi; ++x) v += cs[h][x];
          v *= inv_k;
        }
        score += v;
      }
      score *= inv_n;
    } else {                        // average the SRH sums, then pool
      if (a.pool_type == 0) {
        score = -INFINITY;
        for (int x = lo; x <= hi; ++x) {
          float m = 0.f;
          for (int h = 0; h < nh; ++h) m += cs[h][x];
          score = fmaxf(score, m * inv_n);
        }
      } else {
        score = 0.f;
        for (int x = lo; x <= hi; ++x) {
          float m = 0.f;
          for (int h = 0; h < nh; ++h) m += cs[h][x];
          score += m * inv_n;
        }
        score *= inv_k;
      }
    }
    out[j] = score;
    atomicAdd(&hist_s[hist_bin(__float_as_uint(score))], 1);
  }
}

// Pooling with a compile-time radius RP (kernel 2 RP + 1): each thread pools
// PPT consecutive positions of [c0, p_end) from one register window of
// PPT + 2 RP window sums per SRH (independent LDS reads, positions outside
// the prefix [0, P) padded: -inf for max, 0 for average).  Same arithmetic, in
// the same order, as pool_scores.  The scores go to stage[j - c0] (LDS; the
// caller writes them out with whole-line stores), and runs of equal histogram
// bins (plateaus of max pooling) are added with one atomic.
template <int RP, int NT, int CSW>
__device__ __forceinline__ void pool_scores_r(const ScoreArgs &a, const float (*cs)[CSW],
                                              int nh, int c0, int p_end, int P, float *stage,
                                              int *hist_s) {
  constexpr int PPT = 4;
  constexpr int NV = PPT + 2 * RP;
  const bool is_max = (a.pool_type == 0);
  const float pad = is_max ? -INFINITY : 0.f;
  const float inv_k = 1.f / (float)a.pool_kernel;
  const float inv_n = 1.f / (float)nh;
  for (int j0 = c0 + PPT * (int)threadIdx.x; j0 < p_end; j0 += PPT * NT) {
    float score[PPT];
    if (a.reduce_order == 0) {      // pool each SRH, then average
#pragma unroll
      for (int p = 0; p < PPT; ++p) score[p] = 0.f;
      for (int h = 0; h < nh; ++h) {
        float v[NV];
#pragma unroll
        for (int k = 0; k < NV; ++k) {
          const int x = j0 - RP + k;
          v[k] = (x >= 0 && x < P) ? cs[h][16 + x - c0] : pad;
        }
#pragma unroll
        for (int p = 0; p < PPT; ++p) {
          float m = v[p];
#pragma unroll
          for (int d = 1; d <= 2 * RP; ++d) m = is_max ? fmaxf(m, v[p + d]) : m + v[p + d];
          score[p] += is_max ? m : m * inv_k;
        }
      }
#pragma unroll
      for (int p = 0; p < PPT; ++p) score[p] *= inv_n;
    } else {                        // average the SRH sums, then pool
      float v[NV];
#pragma unroll
      for (int k = 0; k < NV; ++k) {
        const int x = j0 - RP + k;
        if (x >= 0 && x < P) {
          float m = 0.f;
          for (int h = 0; h < nh; ++h) m += cs[h][16 + x - c0];
          v[k] = m * inv_n;
        } else {
          v[k] = pad;
        }
      }
#pragma unroll
      for (int p = 0; p < PPT; ++p) {
        float m = v[p];
#pragma unroll
        for (int d = 1; d <= 2 * RP; ++d) m = is_max ? fmaxf(m, v[p + d]) : m + v[p + d];
        score[p] = is_max ? m : m * inv_k;
      }
    }
    int run_bin = -1, run_n = 0;
#pragma unroll
    for (int p = 0; p < PPT; ++p) {
      if (j0 + p >= p_end) break;
      stage[j0 + p - c0] = score[p];
      const int bin = hist_bin(__float_as_uint(score[p]));
      if (bin != run_bin) {
        if (run_n) atomicAdd(&hist_s[run_bin], run_n);
        run_bin = bin;
        run_n = 0;
      }
      ++run_n;
    }
    if (run_n) atomicAdd(&hist_s[run_bin], run_n);
  }
}

// S4 for one chunk: the compiled radius for the usual kernels (scores staged
// in LDS, then stored a line at a time), the general loop otherwise (or when
// there is no staging buffer).
template <int NT, int CSW>
__device__ __forceinline__ void pool_chunk(const ScoreArgs &a, const float (*cs)[CSW], int nh,
                                           int c0, int p_end, int P, gptr<float> out,
                                           float *stage, int *hist_s) {
  const int rp = (a.pool_kernel - 1) >> 1;
  if (rp > 3 || stage == nullptr) {
    pool_scores<NT, CSW>(a, cs, nh, c0, p_end, P, out, hist_s);
    return;
  }
  switch (rp) {
    case 0: pool_scores_r<0, NT, CSW>(a, cs, nh, c0, p_end, P, stage, hist_s); break;
    case 1: pool_scores_r<1, NT, CSW>(a, cs, nh, c0, p_end, P, stage, hist_s); break;
    case 2: pool_scores_r<2, NT, CSW>(a, cs, nh, c0, p_end, P, stage, hist_s); break;
    default: pool_scores_r<3, NT, CSW>(a, cs, nh, c0, p_end, P, stage, hist_s); break;
  }
  __syncthreads();
  for (int j = c0 + (int)threadIdx.x; j < p_end; j += NT) out[j] = stage[j - c0];
}

// Add a workgroup's LDS histogram to the group's global one (integer atomics:
// the result does not depend on their order).
template <int NT>
__device__ __forceinline__ void flush_hist(const int *hist_s, int *hg) {
  for (int i = threadIdx.x; i < kHistBins; i += NT) {
    const int n = hist_s[i];
    if (n) atomicAdd(&hg[i], n);
  }
}

}  // namespace ckv
