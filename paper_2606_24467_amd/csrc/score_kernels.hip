// Scoring kernels of the CompressKV eviction path (steps S1-S4) for gfx950.
//
// The window softmax (section 3.3, SnapKV-style window of section 4) needs each
// window row's statistics over the whole sequence before any column can be
// normalised, so scoring runs in two kernels over K:
//
//   stats_kernel   S1+S2: per (sequence, KV group, key chunk) it computes the
//                  logits of all SRH window rows against the chunk's keys on
//                  MFMA and reduces them to a per-row partial (ref, sum) with
//                  sum = sum_j exp2(y_j - ref), y = logit * log2(e).
//   colsum_kernel  S2+S3+S4: merges the partials into each row's normaliser,
//                  recomputes the logits of its chunk (plus a 16-key halo on
//                  each side for pooling), sums the normalised probabilities
//                  over the window rows of each SRH, pools along the token axis
//                  in LDS and averages over the SRHs.
//
// Rows of a KV group: SRH h (in head order) owns th = ceil(W/16) row tiles of
// 16 rows; row i < W of the tile set is window query i of that head, the
// padding rows have zero queries and are ignored.
#include "ckv_device.h"

namespace ckv {

// Load one 16-row operand tile of window queries (rows = window positions of
// one SRH) into per-lane slices.  Rows past W are zero.
template <typename T, int D>
__device__ __forceinline__ void load_q_tile(const ScoreArgs &a, int b, int head, int row0,
                                            int c, int quad, uint4 (&out)[Slices<T, D>::n]) {
  const int i = row0 + c;
  if (i < a.W) {
    const char *p = reinterpret_cast<const char *>(a.q) +
                    ((((int64_t)b * a.W + i) * a.Hq + head) * D) * (int64_t)sizeof(T) + 16 * quad;
#pragma unroll
    for (int s = 0; s < Slices<T, D>::n; ++s) out[s] = load16(p + 64 * s);
  } else {
#pragma unroll
    for (int s = 0; s < Slices<T, D>::n; ++s) out[s] = make_uint4(0, 0, 0, 0);
  }
}

// Load the slices of one key row (key index clamped into the sequence).
template <typename T, int D>
__device__ __forceinline__ void load_k_row(const ScoreArgs &a, int s0, int key, int g, int quad,
                                           uint4 (&out)[Slices<T, D>::n]) {
  const char *p = reinterpret_cast<const char *>(a.k) +
                  ((int64_t)(s0 + key) * a.k_stride_tok + (int64_t)g * a.k_stride_head) *
                      (int64_t)sizeof(T) +
                  16 * quad;
#pragma unroll
  for (int s = 0; s < Slices<T, D>::n; ++s) out[s] = load16(p + 64 * s);
}

// ---------------------------------------------------------------------------
// S1+S2 partial statistics.  Grid (max_chunks1, Hkv, batch), 256 threads.
// MFMA operands: A = 16 keys, B = 16 window rows, so lane (quad, c) holds the
// logits of row c against keys 4*quad .. 4*quad+3 of the tile and keeps one
// running (ref, sum) pair per row tile.
// ---------------------------------------------------------------------------
template <typename T, int D, int RTM>
__global__ __launch_bounds__(256) void stats_kernel(const ScoreArgs a) {
  constexpr int NS = Slices<T, D>::n;
  constexpr float kRescale = 30.f;   // rebase the reference when a term would exceed 2^30
  const int chunk = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int s0 = a.cu[b];
  const int L = a.cu[b + 1] - s0;
  const int c0 = chunk * a.chunk1;
  if (c0 >= L) return;                       // uniform for the whole workgroup
  const int c_end = min(L, c0 + a.chunk1);
  const int P = L - a.W;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int c = lane & 15, quad = lane >> 4;
  const int off = a.srh_off[g];
  const int rt_n = (a.srh_off[g + 1] - off) * a.th;

  uint4 qf[RTM][NS];
#pragma unroll
  for (int rt = 0; rt < RTM; ++rt) {
    if (rt < rt_n) {
      load_q_tile<T, D>(a, b, a.srh_head[off + rt / a.th], (rt % a.th) * 16, c, quad, qf[rt]);
    } else {
#pragma unroll
      for (int s = 0; s < NS; ++s) qf[rt][s] = make_uint4(0, 0, 0, 0);
    }
  }
  // row held by this lane in row tile rt: rt*16 + c; its window index:
  float ref[RTM], sum[RTM];
#pragma unroll
  for (int rt = 0; rt < RTM; ++rt) {
    ref[rt] = -INFINITY;
    sum[rt] = 0.f;
  }

  const int ntiles = (c_end - c0 + 15) >> 4;
  uint4 kcur[NS], knext[NS];
  int t = wave;
  if (t < ntiles) load_k_row<T, D>(a, s0, min(c0 + 16 * t + c, L - 1), g, quad, kcur);
  for (; t < ntiles; t += 4) {
    const int base = c0 + 16 * t;
    if (t + 4 < ntiles) load_k_row<T, D>(a, s0, min(base + 64 + c, L - 1), g, quad, knext);
    f32x4 acc[RTM];
#pragma unroll
    for (int rt = 0; rt < RTM; ++rt) {
      acc[rt] = f32x4{0.f, 0.f, 0.f, 0.f};
      if (rt < rt_n) {
#pragma unroll
        for (int s = 0; s < NS; ++s) acc[rt] = mfma_slice<T>(kcur[s], qf[rt][s], acc[rt]);
      }
    }
    // keys of this lane: base + 4*quad + r; masked past the sequence end and,
    // inside the window, after the row's own position (causal).
    const bool masked_tile = (base + 16 > P);
    float d[RTM][4];
    float dmax = -INFINITY;
#pragma unroll
    for (int rt = 0; rt < RTM; ++rt) {
      if (rt >= rt_n) continue;
      const int i = (rt % a.th) * 16 + c;   // window index of this lane's row
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        float x = __builtin_fmaf(acc[rt][r], a.c1, -ref[rt]);
        if (masked_tile) {
          const int j = base + 4 * quad + r;
          const bool ok = (j < L) && (i >= a.W || j <= P + i);
          x = ok ? x : -INFINITY;
        }
        d[rt][r] = x;
        dmax = fmaxf(dmax, x);
      }
    }
    if (__any(dmax > kRescale)) {
      // Rebase a row's reference on the largest new value when a term would
      // exceed 2^kRescale (always the case for the first key of a row).
#pragma unroll
      for (int rt = 0; rt < RTM; ++rt) {
        if (rt >= rt_n) continue;
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
    for (int rt = 0; rt < RTM; ++rt) {
      if (rt >= rt_n) continue;
#pragma unroll
      for (int r = 0; r < 4; ++r) sum[rt] += fast_exp2(d[rt][r]);
    }
#pragma unroll
    for (int s = 0; s < NS; ++s) kcur[s] = knext[s];
  }

  // merge the four quads (same row c, different keys), then the four waves
#pragma unroll
  for (int rt = 0; rt < RTM; ++rt) {
#pragma unroll
    for (int o = 16; o <= 32; o <<= 1) {
      float ro = __shfl_xor(ref[rt], o);
      float so = __shfl_xor(sum[rt], o);
      merge_stats(ref[rt], sum[rt], ro, so);
    }
  }
  __shared__ float2 part[4][RTM * 16];
  if (quad == 0) {
#pragma unroll
    for (int rt = 0; rt < RTM; ++rt) part[wave][rt * 16 + c] = make_float2(ref[rt], sum[rt]);
  }
  __syncthreads();
  const int tid = threadIdx.x;
  if (tid < rt_n * 16) {
    float r0 = part[0][tid].x, s_0 = part[0][tid].y;
#pragma unroll
    for (int w = 1; w < 4; ++w) merge_stats(r0, s_0, part[w][tid].x, part[w][tid].y);
    a.stats[(((int64_t)b * a.Hkv + g) * a.max_chunks1 + chunk) * a.row_slots + tid] =
        make_float2(r0, s_0);
  }
}

// ---------------------------------------------------------------------------
// S2+S3+S4.  Grid (max_chunks2, Hkv, batch), 256 threads.
// MFMA operands: A = 16 window rows, B = 16 keys, so lane (quad, c) holds
// rows 4*quad .. 4*quad+3 of the tile against key c.
// ---------------------------------------------------------------------------
template <typename T, int D, int RTM>
__global__ __launch_bounds__(256) void colsum_kernel(const ScoreArgs a) {
  constexpr int NS = Slices<T, D>::n;
  constexpr int kMaxChunk2 = 1024;
  constexpr int kMaxSrh = RTM;   // th >= 1
  const int chunk = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
  const int s0 = a.cu[b];
  const int L = a.cu[b + 1] - s0;
  const int c0 = chunk * a.chunk2;
  if (c0 >= L) return;
  const int c_end = min(L, c0 + a.chunk2);
  const int P = L - a.W;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int c = lane & 15, quad = lane >> 4;
  const int tid = threadIdx.x;
  const int off = a.srh_off[g];
  const int nh = a.srh_off[g + 1] - off;
  const int rt_n = nh * a.th;
  float *out = a.scores + (int64_t)g * a.T + s0;

  // Window positions of this chunk are always kept: +inf.
  for (int j = max(c0, P) + tid; j < c_end; j += 256) out[j] = INFINITY;
  if (c0 >= P) return;                        // no prefix key in this chunk
  const int p_end = min(c_end, P);

  // Row normalisers: bias = ref + log2(sum) over all chunks of the statistics pass.
  __shared__ float bias_s[RTM * 16];
  if (tid < rt_n * 16) {
    const int nc1 = (L + a.chunk1 - 1) / a.chunk1;
    const float2 *st = a.stats + ((int64_t)b * a.Hkv + g) * a.max_chunks1 * a.row_slots + tid;
    float m = -INFINITY;
    for (int k = 0; k < nc1; ++k) m = fmaxf(m, st[(int64_t)k * a.row_slots].x);
    float sm = 0.f;
    for (int k = 0; k < nc1; ++k) {
      float2 v = st[(int64_t)k * a.row_slots];
      sm += v.y * fast_exp2(v.x - m);
    }
    const int i = (tid % (16 * a.th));
    bias_s[tid] = (i < a.W) ? m + fast_log2(sm) : INFINITY;
  } else if (tid < RTM * 16) {
    bias_s[tid] = INFINITY;
  }

  uint4 qf[RTM][NS];
#pragma unroll
  for (int rt = 0; rt < RTM; ++rt) {
    if (rt < rt_n) {
      load_q_tile<T, D>(a, b, a.srh_head[off + rt / a.th], (rt % a.th) * 16, c, quad, qf[rt]);
    } else {
#pragma unroll
      for (int s = 0; s < NS; ++s) qf[rt][s] = make_uint4(0, 0, 0, 0);
    }
  }
  __syncthreads();
  float bias[RTM][4];
#pragma unroll
  for (int rt = 0; rt < RTM; ++rt)
#pragma unroll
    for (int r = 0; r < 4; ++r) bias[rt][r] = bias_s[rt * 16 + 4 * quad + r];

  // Column sums of the chunk plus one 16-key halo tile on each side.
  // cs[h][16 + x] holds the window sum of SRH h at key c0 + x.
  __shared__ float cs[kMaxSrh][kMaxChunk2 + 32];
  const int ntiles = (p_end - c0 + 15) >> 4;        // tiles e = 0 .. ntiles-1
  const int e_lo = (c0 > 0) ? -1 : 0;
  const int e_hi = (c0 + 16 * ntiles < P) ? ntiles : ntiles - 1;
  for (int e = e_lo + wave; e <= e_hi; e += 4) {
    const int base = c0 + 16 * e;
    uint4 kf[NS];
    load_k_row<T, D>(a, s0, min(base + c, L - 1), g, quad, kf);
    f32x4 acc[RTM];
#pragma unroll
    for (int rt = 0; rt < RTM; ++rt) {
      acc[rt] = f32x4{0.f, 0.f, 0.f, 0.f};
      if (rt < rt_n) {
#pragma unroll
        for (int s = 0; s < NS; ++s) acc[rt] = mfma_slice<T>(qf[rt][s], kf[s], acc[rt]);
      }
    }
    // Sum the normalised probabilities over the window rows of each SRH:
    // in-lane over the 4 rows and the SRH's row tiles, then across the quads.
    int hh = 0;
    float v = 0.f;
#pragma unroll
    for (int rt = 0; rt < RTM; ++rt) {
      if (rt >= rt_n) continue;
#pragma unroll
      for (int r = 0; r < 4; ++r) v += fast_exp2(__builtin_fmaf(acc[rt][r], a.c1, -bias[rt][r]));
      if ((a.head_end_mask >> rt) & 1u) {
        v += __shfl_xor(v, 16);
        v += __shfl_xor(v, 32);
        if (quad == (hh & 3)) cs[hh][16 + 16 * e + c] = v;
        v = 0.f;
        ++hh;
      }
    }
  }
  __syncthreads();

  // Pooling along the token axis (positions clipped to the prefix [0, P)),
  // then the mean over the group's SRHs.
  const int rp = (a.pool_kernel - 1) >> 1;
  const float inv_k = 1.f / (float)a.pool_kernel;
  const float inv_n = 1.f / (float)nh;
  for (int j = c0 + tid; j < p_end; j += 256) {
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
  }
}

// ---------------------------------------------------------------------------
// Host-side launchers (called by the C ABI after validation).
// ---------------------------------------------------------------------------
template <typename T, int D, int RTM>
static hipError_t launch_score_t(const ScoreArgs &a, int batch, hipStream_t stream) {
  dim3 block(256);
  hipLaunchKernelGGL((stats_kernel<T, D, RTM>), dim3(a.max_chunks1, a.Hkv, batch), block, 0,
                     stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((colsum_kernel<T, D, RTM>), dim3(a.max_chunks2, a.Hkv, batch), block, 0,
                     stream, a);
  return hipGetLastError();
}

template <typename T, int D>
static hipError_t launch_score_d(const ScoreArgs &a, int rt_max, int batch, hipStream_t stream) {
  if (rt_max <= 2) return launch_score_t<T, D, 2>(a, batch, stream);
  if (rt_max <= 4) return launch_score_t<T, D, 4>(a, batch, stream);
  if (rt_max <= 8) return launch_score_t<T, D, 8>(a, batch, stream);
  return launch_score_t<T, D, 12>(a, batch, stream);
}

hipError_t launch_score(const ScoreArgs &a, int dtype_bf16, int head_dim, int rt_max, int batch,
                        hipStream_t stream) {
  if (dtype_bf16) {
    return head_dim == 64 ? launch_score_d<__bf16, 64>(a, rt_max, batch, stream)
                          : launch_score_d<__bf16, 128>(a, rt_max, batch, stream);
  }
  return head_dim == 64 ? launch_score_d<float, 64>(a, rt_max, batch, stream)
                        : launch_score_d<float, 128>(a, rt_max, batch, stream);
}

}  // namespace ckv
