// Eviction error of a layer (section 3.4, equations 2-4): over decoding steps,
// ||W_O (A_full - A_comp)||_F / (||W_O A_full||_F + eps), where A is the
// attention of the step's queries over the full KV cache or over the compact
// cache that the eviction path wrote.
//
//   dec_attn_kernel     split-K attention of every (sequence, group, cache):
//                       the group's rows (decoding step x query head of the
//                       group) against one 512-key chunk, QK^T on MFMA, online
//                       softmax in LDS, P.V on fp32 MFMA; partial (max, sum, O)
//   dec_combine_kernel  merges the chunks of every row into A (fp32)
//   dec_proj_kernel     y = W_O x for x = A_full and A_full - A_comp on fp32
//                       MFMA (16 rows of W_O per workgroup, 16 waves on
//                       sixteenths of its columns); per-workgroup sums of y^2
//   dec_error_kernel    the per-step norms, their ratios and the layer sum
//
// The kernels take a block of at most kMaxVectors (sequence, step) vectors
// whose rows per group (steps x query heads of the group) fit kMaxDecRows;
// longer decodes and larger batches run block after block, each adding its
// ratios to the sum.  Every reduction runs in a fixed order, so the result is
// deterministic.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>

#include "../../include/compresskv_offline.h"
#include "api_common.h"
#include "score_common.h"

namespace ckv {

constexpr int kDecChunk = 512;   // keys per attention workgroup (eight softmax steps)
constexpr int kDecSub = 64;      // keys per softmax step inside it (one tile per wave)
constexpr int kProjRows = 16;    // W_O rows per projection workgroup
constexpr int kProjWaves = 16;   // waves per projection workgroup, each on HD / 16 columns
constexpr int kMaxDecRows = 64;  // decoding steps x query heads per group, per block
constexpr int kMaxVectors = 32;  // sequences x decoding steps, per block

// One block: sequences b0 .. b0 + batch - 1, steps t0 .. t0 + T - 1; the
// partials and A are indexed by the block's own sequence and step.
struct DecArgs {
  const char *q;                 // [all sequences][q_T][Hq][D]
  const char *k, *v;             // full caches, byte strides below
  const char *k_out, *v_out;     // compact caches [all sequences][Hkv][B][D]
  const int32_t *cu;
  float2 *part_ml;               // [2][batch][Hkv][n_chunks][64] (max, sum), log2 domain
  float *part_o;                 // [2][batch][Hkv][n_chunks][64][D]
  float *a;                      // [2][batch][T][Hq][D]
  int64_t k_st, k_sh, v_st, v_sh;
  int T, Hq, Hkv, G, B, batch, R, n_chunks;
  int b0, t0, q_T;               // the block's first sequence and step; steps in q
  float c1;                      // softmax scale * log2(e)
};

// Cache `cache` (0 full, 1 compact) of sequence b, group g: keys and the byte
// address of key row j of K (or V).
struct DecCache {
  int n_keys;
  const char *kb, *vb;
  int64_t k_row, v_row;          // byte stride between rows
};

template <typename T, int D>
__device__ __forceinline__ DecCache dec_cache(const DecArgs &a, int cache, int b, int g) {
  DecCache c;
  const int s0 = a.cu[b], L = a.cu[b + 1] - s0;
  if (cache == 0) {
    c.n_keys = L;
    c.kb = a.k + (int64_t)s0 * a.k_st + (int64_t)g * a.k_sh;
    c.vb = a.v + (int64_t)s0 * a.v_st + (int64_t)g * a.v_sh;
    c.k_row = a.k_st;
    c.v_row = a.v_st;
  } else {
    c.n_keys = min(L, a.B);   // the eviction path keeps min(L, B) rows, in its first entries
    const int64_t base = ((int64_t)b * a.Hkv + g) * a.B * D * (int64_t)sizeof(T);
    c.kb = a.k_out + base;
    c.vb = a.v_out + base;
    c.k_row = c.v_row = D * (int64_t)sizeof(T);
  }
  return c;
}

// Grid (n_chunks, Hkv, batch * 2), 256 threads.  Rows r = t * G + hh (step t,
// head g * G + hh); RT = ceil(R / 16) row tiles, padding rows have zero
// queries.  The P.V step runs on v_mfma_f32_16x16x4_f32 with fp32
// probabilities and V converted exactly to fp32: wave w owns the output
// tiles of every row tile and the column tiles w*CTW .. +CTW (lane (quad, c)
// holds rows 4*quad .. +3 of a tile against column c).
template <typename T, int D, int RT>
__global__ __launch_bounds__(256) void dec_attn_kernel(const DecArgs a) {
  constexpr int NS = Slices<T, D>::n, U4 = QLayout<T, D>::U4, STRIDE = QLayout<T, D>::STRIDE;
  constexpr int RP = RT * 16;                  // rows with padding
  constexpr int CTW = D / 16 / 4;              // column tiles per wave in the P.V step
  constexpr int ZS = kDecSub + 1;              // padded row of the logits buffer
  static_assert(CTW >= 1 && D % 64 == 0, "column tiles");
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int c = lane & 15, quad = lane >> 4;
  const int g = blockIdx.y, b = (int)blockIdx.z >> 1, cache = (int)blockIdx.z & 1;
  const DecCache cc = dec_cache<T, D>(a, cache, a.b0 + b, g);
  const int c0 = (int)blockIdx.x * kDecChunk;
  if (c0 >= cc.n_keys) return;   // uniform
  const int c_end = min(cc.n_keys, c0 + kDecChunk);

  __shared__ uint4 q_lds[RP * STRIDE];
  __shared__ float zs[RP * ZS];                 // logits, then probabilities
  __shared__ uint4 vs4[kDecSub * D * sizeof(T) / 16];   // the step's V rows
  const T *vs = reinterpret_cast<const T *>(vs4);
  __shared__ float m_s[RP], l_s[RP], alpha_s[RP];

  // queries of the group's rows
  for (int i = tid; i < RP * U4; i += 256) {
    const int r = i / U4, u = i - r * U4;
    uint4 val = make_uint4(0, 0, 0, 0);
    if (r < a.R) {
      const int t = r / a.G, h = g * a.G + (r - t * a.G);
      val = load16(to_global(a.q) +
                   (((int64_t)(a.b0 + b) * a.q_T + a.t0 + t) * a.Hq + h) * (D * (int64_t)sizeof(T)) +
                   16 * u);
    }
    q_lds[r * STRIDE + u] = val;
  }
  if (tid < RP) {
    m_s[tid] = -INFINITY;
    l_s[tid] = 0.f;
  }
  __syncthreads();
  uint4 qreg[RegTiles<T, D, RT>::n][NS];
#pragma unroll
  for (int rt = 0; rt < RegTiles<T, D, RT>::v; ++rt)
#pragma unroll
    for (int s = 0; s < NS; ++s) qreg[rt][s] = q_frag<T, D>(q_lds, rt, s, c, quad);

  f32x4 acc[RT][CTW];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int ct = 0; ct < CTW; ++ct) acc[rt][ct] = f32x4{0.f, 0.f, 0.f, 0.f};

  // The K fragments and V rows of a step are loaded into registers one step
  // ahead: the next step's loads are in flight during this step's softmax and
  // P.V.
  constexpr int KT = kDecSub / 64;                   // key tiles per wave and step
  constexpr int V4 = D * (int)sizeof(T) / 16;        // 16-byte units per V row
  constexpr int VPT = kDecSub * V4 / 256;            // V units per thread and step
  static_assert(kDecSub * V4 % 256 == 0, "V units");
  uint4 kf[KT][NS], vr[VPT];
  auto issue = [&](int k0) {
#pragma unroll
    for (int i = 0; i < KT; ++i) {
      const int key = min(k0 + 16 * (wave + 4 * i) + c, cc.n_keys - 1);
      const gptr<const char> p = to_global(cc.kb) + key * cc.k_row + 16 * quad;
#pragma unroll
      for (int s = 0; s < NS; ++s) kf[i][s] = load16(p + 64 * s);
    }
#pragma unroll
    for (int u = 0; u < VPT; ++u) {
      const int idx = tid + 256 * u, j = idx / V4, uu = idx - j * V4;
      const int key = min(k0 + j, cc.n_keys - 1);
      vr[u] = load16(to_global(cc.vb) + key * cc.v_row + 16 * uu);
    }
  };
  issue(c0);
  for (int k0 = c0; k0 < c_end; k0 += kDecSub) {
    // S: logits of the step's key tiles (KT per wave), in log2 units
#pragma unroll
    for (int i = 0; i < KT; ++i) {
      const int e = wave + 4 * i;
      f32x4 lg[RT];
      tile_logits_all<T, D, RT, true>(kf[i], qreg, q_lds, c, quad, lg);
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int j = 16 * e + 4 * quad + r;
          zs[(rt * 16 + c) * ZS + j] = (k0 + j < c_end) ? lg[rt][r] * a.c1 : -INFINITY;
        }
    }
    // V rows of the step
#pragma unroll
    for (int u = 0; u < VPT; ++u) vs4[tid + 256 * u] = vr[u];
    if (k0 + kDecSub < c_end) issue(k0 + kDecSub);   // uniform
    __syncthreads();
    // online softmax: four threads per row, kDecSub / 4 keys each
    {
      constexpr int KPT = kDecSub / 4;
      const int r = tid >> 2, part = tid & 3;
      if (r < RP) {
        float* zr = zs + r * ZS + KPT * part;
        float mx = -INFINITY;
        for (int j = 0; j < KPT; ++j) mx = fmaxf(mx, zr[j]);
        mx = fmaxf(mx, __shfl_xor(mx, 1));
        mx = fmaxf(mx, __shfl_xor(mx, 2));
        const float m_old = m_s[r];
        const float m_new = fmaxf(m_old, mx);
        // a row with no visible key yet keeps zero weight
        const float alpha = (m_new == -INFINITY) ? 1.f : fast_exp2(m_old - m_new);
        float sm = 0.f;
        for (int j = 0; j < KPT; ++j) {
          const float p = (m_new == -INFINITY) ? 0.f : fast_exp2(zr[j] - m_new);
          zr[j] = p;
          sm += p;
        }
        sm += __shfl_xor(sm, 1);
        sm += __shfl_xor(sm, 2);
        // the four threads of a row hold the same values; the first writes
        if (part == 0) {
          m_s[r] = m_new;
          l_s[r] = l_s[r] * alpha + sm;
          alpha_s[r] = alpha;
        }
      }
    }
    __syncthreads();
    // O = alpha * O + P.V: keys 4 j + quad of the step per MFMA (keys past the
    // chunk have p = 0)
#pragma unroll
    for (int rt = 0; rt < RT; ++rt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float al = alpha_s[rt * 16 + 4 * quad + r];
#pragma unroll
        for (int ct = 0; ct < CTW; ++ct) acc[rt][ct][r] *= al;
      }
#pragma unroll 4
    for (int j = 0; j < kDecSub / 4; ++j) {
      const int key = 4 * j + quad;
      float vv[CTW];
#pragma unroll
      for (int ct = 0; ct < CTW; ++ct) vv[ct] = (float)vs[key * D + 16 * (wave * CTW + ct) + c];
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        const float p = zs[(rt * 16 + c) * ZS + key];
#pragma unroll
        for (int ct = 0; ct < CTW; ++ct)
          acc[rt][ct] = __builtin_amdgcn_mfma_f32_16x16x4f32(p, vv[ct], acc[rt][ct], 0, 0, 0);
      }
    }
    __syncthreads();   // zs and vs are rewritten by the next step
  }
  // partials of this chunk
  const int64_t slot = (((int64_t)cache * a.batch + b) * a.Hkv + g) * a.n_chunks + blockIdx.x;
  if (tid < a.R) a.part_ml[slot * kMaxDecRows + tid] = make_float2(m_s[tid], l_s[tid]);
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int row = rt * 16 + 4 * quad + r;
      if (row < a.R) {
        float *o = a.part_o + (slot * kMaxDecRows + row) * D;
#pragma unroll
        for (int ct = 0; ct < CTW; ++ct) o[16 * (wave * CTW + ct) + c] = acc[rt][ct][r];
      }
    }
}

// Grid (R, Hkv, batch * 2), D threads: A of row r of the group from its
// chunks.  The chunk maxima and weights are formed in parallel (LDS), the
// weighted sums run over the chunks in order (thread d: column d).
template <int D>
__global__ __launch_bounds__(D) void dec_combine_kernel(const DecArgs a) {
  constexpr int kMaxCh = 1024;   // chunks per pass of the weight table
  __shared__ float w_s[kMaxCh];
  __shared__ float red[D];
  const int r = blockIdx.x, g = blockIdx.y, b = (int)blockIdx.z >> 1, cache = (int)blockIdx.z & 1;
  const int d = threadIdx.x;
  const int L = a.cu[a.b0 + b + 1] - a.cu[a.b0 + b];
  const int n_keys = cache == 0 ? L : min(L, a.B);
  const int nch = (n_keys + kDecChunk - 1) / kDecChunk;
  const int64_t slot0 = (((int64_t)cache * a.batch + b) * a.Hkv + g) * a.n_chunks;
  // the row's maximum over its chunks: per thread over chunks d, d + D, ...,
  // then a tree in LDS (max is exact in any order)
  float M = -INFINITY;
  for (int ch = d; ch < nch; ch += D) M = fmaxf(M, a.part_ml[(slot0 + ch) * kMaxDecRows + r].x);
  red[d] = M;
  __syncthreads();
  for (int h = D / 2; h > 0; h >>= 1) {
    if (d < h) red[d] = fmaxf(red[d], red[d + h]);
    __syncthreads();
  }
  M = red[0];
  float lsum = 0.f, o = 0.f;
  for (int c0 = 0; c0 < nch; c0 += kMaxCh) {
    const int n = min(kMaxCh, nch - c0);
    __syncthreads();
    for (int ch = d; ch < n; ch += D)
      w_s[ch] = fast_exp2(a.part_ml[(slot0 + c0 + ch) * kMaxDecRows + r].x - M);
    __syncthreads();
    const float *po = a.part_o + ((slot0 + c0) * kMaxDecRows + r) * D + d;
#pragma unroll 8
    for (int ch = 0; ch < n; ++ch) o += po[(int64_t)ch * kMaxDecRows * D] * w_s[ch];
    // every thread forms the same sum of the chunk sums, in chunk order
    for (int ch = 0; ch < n; ++ch)
      lsum += a.part_ml[(slot0 + c0 + ch) * kMaxDecRows + r].y * w_s[ch];
  }
  const int t = r / a.G, h = g * a.G + (r - t * a.G);
  a.a[((((int64_t)cache * a.batch + b) * a.T + t) * a.Hq + h) * D + d] = o / lsum;
}

struct ProjArgs {
  const char *w_o;          // [d_model][HD], dtype T
  const float *a;           // [2][NV][HD]: A_full, A_comp
  float *part_ss;           // [n_wg][2][kMaxVectors]: sums of y_full^2, y_diff^2 over the
                            // workgroup's rows of W_O
  int d_model, HD, NV;
};

// Grid (ceil(d_model / 16)), 1024 threads.  The vectors are the rows of
// X = [A_full (NV rows); A_full - A_comp (NV rows); zeros], in XT tiles of 16;
// wave w computes Y = X W_O^T over the w-th sixteenth of the columns for
// every X tile and the workgroup's 16 rows of W_O with v_mfma_f32_16x16x4_f32
// (MFMA operands as in the scoring kernels: lane (quad, c) holds floats
// 16 s + 4 quad .. +3 of row c of each tile).  The sixteen partial products
// are added in wave order, then y^2 is summed over the 16 rows of W_O (lanes
// c, fixed butterfly).
template <typename T, int XT>
__global__ __launch_bounds__(64 * kProjWaves) void dec_proj_kernel(const ProjArgs p) {
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int c = lane & 15, quad = lane >> 4;
  const int o = (int)blockIdx.x * kProjRows + c;            // this lane's row of W_O
  const bool o_ok = o < p.d_model;
  const T *wr = reinterpret_cast<const T *>(p.w_o) + (int64_t)(o_ok ? o : 0) * p.HD;
  const float *xf[XT], *xc[XT];
  int kind[XT];
#pragma unroll
  for (int x = 0; x < XT; ++x) {
    const int n = 16 * x + c;                                 // this lane's row of X tile x
    kind[x] = n < p.NV ? 0 : (n < 2 * p.NV ? 1 : 2);          // full, difference, padding
    const int v = kind[x] == 0 ? n : (kind[x] == 1 ? n - p.NV : 0);
    xf[x] = p.a + (int64_t)v * p.HD;
    xc[x] = p.a + (int64_t)(p.NV + v) * p.HD;
  }
  f32x4 acc[XT];
#pragma unroll
  for (int x = 0; x < XT; ++x) acc[x] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int qw = p.HD / kProjWaves;                           // columns per wave
  const int k_end = (wave + 1) * qw;
  // X tile x's four floats at column k (row as set above), the difference
  // rows formed here
  auto x_at = [&](int x, int k) {
    float4 xv = *reinterpret_cast<const float4 *>(xf[x] + k);
    if (kind[x] == 1) {
      const float4 y = *reinterpret_cast<const float4 *>(xc[x] + k);
      xv = make_float4(xv.x - y.x, xv.y - y.y, xv.z - y.z, xv.w - y.w);
    } else if (kind[x] == 2) {
      xv = make_float4(0.f, 0.f, 0.f, 0.f);
    }
    return xv;
  };
  auto w_at = [&](int k) {   // four elements of this lane's row of W_O at column k
    float4 wv;
    if constexpr (sizeof(T) == 2) {
      const uint2 raw = *reinterpret_cast<const uint2 *>(wr + k);
      wv = make_float4(__uint_as_float(raw.x << 16), __uint_as_float(raw.x & 0xFFFF0000u),
                       __uint_as_float(raw.y << 16), __uint_as_float(raw.y & 0xFFFF0000u));
    } else {
      wv = *reinterpret_cast<const float4 *>(wr + k);
    }
    return o_ok ? wv : make_float4(0.f, 0.f, 0.f, 0.f);
  };
  // 64 columns per trip: lane (quad, c) takes the 16 consecutive columns
  // k0 + 16 quad .. + 15 of its row of W_O (a whole 32-byte or 64-byte run)
  // and of its X rows, four MFMA steps of 4 columns each (the products are
  // summed over the columns, so which 4 columns a step takes is free as long
  // as W_O and X agree)
  int k0 = wave * qw;
  for (; k0 + 64 <= k_end; k0 += 64) {
    const int kq = k0 + 16 * quad;
    float4 wv[4];
#pragma unroll
    for (int st = 0; st < 4; ++st) wv[st] = w_at(kq + 4 * st);
#pragma unroll
    for (int x = 0; x < XT; ++x) {
#pragma unroll
      for (int st = 0; st < 4; ++st)
        acc[x] = mfma_slice<float>(__builtin_bit_cast(uint4, x_at(x, kq + 4 * st)),
                                   __builtin_bit_cast(uint4, wv[st]), acc[x]);
    }
  }
  // the rest in steps of 16 columns (lane quad on columns k0 + 4 quad .. + 3)
  for (; k0 < k_end; k0 += 16) {
    const float4 wv = w_at(k0 + 4 * quad);
#pragma unroll
    for (int x = 0; x < XT; ++x)
      acc[x] = mfma_slice<float>(__builtin_bit_cast(uint4, x_at(x, k0 + 4 * quad)),
                                 __builtin_bit_cast(uint4, wv), acc[x]);
  }
  __shared__ f32x4 part[kProjWaves][XT][64];
#pragma unroll
  for (int x = 0; x < XT; ++x) part[wave][x][lane] = acc[x];
  __syncthreads();
  // wave x < XT finishes X tile x: the partial products in wave order, then
  // the squares
  if (wave < XT) {
    f32x4 y = part[0][wave][lane];
#pragma unroll
    for (int w = 1; w < kProjWaves; ++w) y = y + part[w][wave][lane];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      float sq = y[r] * y[r];
#pragma unroll
      for (int m = 1; m < 16; m <<= 1) sq += __shfl_xor(sq, m);
      const int row = 16 * wave + 4 * quad + r;
      if (c == 0 && row < 2 * p.NV)
        p.part_ss[((int64_t)blockIdx.x * 2 + (row < p.NV ? 0 : 1)) * kMaxVectors +
                  (row < p.NV ? row : row - p.NV)] = sq;
    }
  }
}

// One workgroup of kMaxVectors waves' worth of lanes: wave n sums vector n's
// squares over the projection workgroups (lane l: workgroups l, l + 64, ...
// in order, then a fixed butterfly), forms the ratio, and thread 0 adds the
// ratios in vector order, to zero (first block) or to the sum so far.
__global__ __launch_bounds__(64 * kMaxVectors / 2) void dec_error_kernel(const float *part_ss,
                                                                        int n_wg, int NV,
                                                                        float eps, int first,
                                                                        float *err) {
  __shared__ float ratio[kMaxVectors];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int n = wave; n < NV; n += blockDim.x / 64) {
    float sf = 0.f, sd = 0.f;
    for (int w = lane; w < n_wg; w += 64) {
      sf += part_ss[((int64_t)w * 2 + 0) * kMaxVectors + n];
      sd += part_ss[((int64_t)w * 2 + 1) * kMaxVectors + n];
    }
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) {
      sf += __shfl_xor(sf, m);
      sd += __shfl_xor(sd, m);
    }
    if (lane == 0) ratio[n] = sqrtf(sd) / (sqrtf(sf) + eps);
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float e = first ? 0.f : err[0];
    for (int n = 0; n < NV; ++n) e += ratio[n];
    err[0] = e;
  }
}

template <typename T, int D>
static void launch_dec_t(const DecArgs &a, const ProjArgs &pa, int rt, int n_wg, float eps,
                         bool first, float *err, hipStream_t s) {
  const dim3 g1(a.n_chunks, a.Hkv, a.batch * 2);
  switch (rt) {
    case 1: hipLaunchKernelGGL((dec_attn_kernel<T, D, 1>), g1, dim3(256), 0, s, a); break;
    case 2: hipLaunchKernelGGL((dec_attn_kernel<T, D, 2>), g1, dim3(256), 0, s, a); break;
    case 3: hipLaunchKernelGGL((dec_attn_kernel<T, D, 3>), g1, dim3(256), 0, s, a); break;
    default: hipLaunchKernelGGL((dec_attn_kernel<T, D, 4>), g1, dim3(256), 0, s, a); break;
  }
  hipLaunchKernelGGL((dec_combine_kernel<D>), dim3(a.R, a.Hkv, a.batch * 2), dim3(D), 0, s, a);
  switch ((2 * pa.NV + 15) / 16) {
    case 1: hipLaunchKernelGGL((dec_proj_kernel<T, 1>), dim3(n_wg), dim3(64 * kProjWaves), 0, s, pa); break;
    case 2: hipLaunchKernelGGL((dec_proj_kernel<T, 2>), dim3(n_wg), dim3(64 * kProjWaves), 0, s, pa); break;
    case 3: hipLaunchKernelGGL((dec_proj_kernel<T, 3>), dim3(n_wg), dim3(64 * kProjWaves), 0, s, pa); break;
    default: hipLaunchKernelGGL((dec_proj_kernel<T, 4>), dim3(n_wg), dim3(64 * kProjWaves), 0, s, pa); break;
  }
  hipLaunchKernelGGL(dec_error_kernel, dim3(1), dim3(64 * kMaxVectors / 2), 0, s, pa.part_ss, n_wg,
                     pa.NV, eps, first ? 1 : 0, err);
}

}  // namespace ckv

namespace {

using ckv_api::fail;
using ckv_api::ok;

struct DecPlan {
  int TS = 0, BS = 0;      // steps and sequences per block
  int R = 0, rt = 0, n_chunks = 0, n_wg = 0, NV = 0, lmax = 0;   // of a full block
  size_t ml_off = 0, o_off = 0, a_off = 0, ss_off = 0, total = 0;
};

size_t round256(size_t x) { return (x + 255) / 256 * 256; }

int check_error_problem(const ckv_problem *p, const ckv_error_problem *e, DecPlan &pl) {
  if (!p || !e) return fail(CKV_INVALID_ARGUMENT, "problem is NULL");
  if (p->batch < 1 || p->n_kv_heads < 1 || p->n_q_heads < 1 ||
      p->n_q_heads % p->n_kv_heads != 0)
    return fail(CKV_INVALID_ARGUMENT, "batch >= 1 and n_q_heads a multiple of n_kv_heads");
  if (p->n_kv_heads > ckv::kMaxKvHeads)
    return fail(CKV_UNSUPPORTED, "at most %d KV heads", ckv::kMaxKvHeads);
  if (p->head_dim != 64 && p->head_dim != 128)
    return fail(CKV_UNSUPPORTED, "head_dim must be 64 or 128 (got %d)", p->head_dim);
  if (p->dtype != CKV_F32 && p->dtype != CKV_BF16)
    return fail(CKV_UNSUPPORTED, "dtype must be CKV_F32 or CKV_BF16");
  if (!std::isfinite(p->scale)) return fail(CKV_INVALID_ARGUMENT, "scale must be finite");
  if (!p->cu_seqlens || !p->cu_seqlens_host)
    return fail(CKV_INVALID_ARGUMENT, "cu_seqlens and cu_seqlens_host are both required");
  if (p->cu_seqlens_host[0] != 0) return fail(CKV_INVALID_ARGUMENT, "cu_seqlens[0] must be 0");
  const int es = p->dtype == CKV_BF16 ? 2 : 4;
  const int64_t strides[4] = {p->k_stride_tok, p->k_stride_head, p->v_stride_tok, p->v_stride_head};
  for (int i = 0; i < 4; ++i)
    if (strides[i] < 1 || (strides[i] * es) % 16 != 0)
      return fail(CKV_UNSUPPORTED, "K/V strides must be >= 1 and multiples of 16 bytes");
  if (e->n_steps < 1) return fail(CKV_INVALID_ARGUMENT, "n_steps must be >= 1");
  if (e->d_model < 1) return fail(CKV_INVALID_ARGUMENT, "d_model must be >= 1");
  if (e->budget < 1) return fail(CKV_INVALID_ARGUMENT, "budget must be >= 1");
  if (!(e->eps >= 0.f) || !std::isfinite(e->eps))
    return fail(CKV_INVALID_ARGUMENT, "eps must be finite and >= 0");
  const int G = p->n_q_heads / p->n_kv_heads;
  if (G > ckv::kMaxDecRows)
    return fail(CKV_UNSUPPORTED, "n_q_heads / n_kv_heads must be <= %d", ckv::kMaxDecRows);
  pl.TS = std::min({ckv::kMaxDecRows / G, ckv::kMaxVectors, e->n_steps});
  pl.BS = std::min(p->batch, ckv::kMaxVectors / pl.TS);
  pl.R = pl.TS * G;
  pl.NV = pl.BS * pl.TS;
  if ((p->n_q_heads * p->head_dim) % 256 != 0)
    return fail(CKV_UNSUPPORTED, "n_q_heads * head_dim must be a multiple of 256");
  pl.lmax = 0;
  for (int b = 0; b < p->batch; ++b) {
    const int L = p->cu_seqlens_host[b + 1] - p->cu_seqlens_host[b];
    if (L < 1) return fail(CKV_INVALID_ARGUMENT, "sequence %d is empty or cu_seqlens decreasing", b);
    pl.lmax = std::max(pl.lmax, L);
  }
  pl.rt = (pl.R + 15) / 16;
  pl.n_chunks = (pl.lmax + ckv::kDecChunk - 1) / ckv::kDecChunk;
  pl.n_wg = (e->d_model + ckv::kProjRows - 1) / ckv::kProjRows;
  const size_t slots = (size_t)2 * pl.BS * p->n_kv_heads * pl.n_chunks * ckv::kMaxDecRows;
  pl.ml_off = 0;
  pl.o_off = round256(slots * sizeof(float2));
  pl.a_off = pl.o_off + round256(slots * p->head_dim * sizeof(float));
  pl.ss_off = pl.a_off +
              round256((size_t)2 * pl.NV * p->n_q_heads * p->head_dim * sizeof(float));
  pl.total = pl.ss_off + round256((size_t)pl.n_wg * 2 * ckv::kMaxVectors * sizeof(float));
  return CKV_OK;
}

}  // namespace

extern "C" {

size_t compresskv_layer_error_workspace_bytes(const ckv_problem *p, const ckv_error_problem *e) {
  DecPlan pl;
  if (check_error_problem(p, e, pl)) return 0;
  ok();
  return pl.total;
}

int compresskv_layer_error(const ckv_problem *p, const ckv_error_problem *e, const void *q_dec,
                           const void *k, const void *v, const void *k_out, const void *v_out,
                           const void *w_o, float *err, void *ws, size_t ws_bytes,
                           void *stream) {
  DecPlan pl;
  int st;
  if ((st = check_error_problem(p, e, pl))) return st;
  const void *ptrs[] = {q_dec, k, v, k_out, v_out, w_o};
  const char *names[] = {"q_dec", "k", "v", "k_out", "v_out", "w_o"};
  for (int i = 0; i < 6; ++i) {
    if (!ptrs[i]) return fail(CKV_INVALID_ARGUMENT, "%s is NULL", names[i]);
    if (!ckv_api::aligned(ptrs[i], 16))
      return fail(CKV_UNSUPPORTED, "%s must be 16-byte aligned", names[i]);
  }
  if (!err) return fail(CKV_INVALID_ARGUMENT, "err is NULL");
  if (!ckv_api::aligned(err, 4)) return fail(CKV_UNSUPPORTED, "err must be 4-byte aligned");
  if (ws_bytes < pl.total)
    return fail(CKV_WORKSPACE_TOO_SMALL, "workspace of %zu bytes, %zu needed", ws_bytes, pl.total);
  if (!ws) return fail(CKV_INVALID_ARGUMENT, "workspace is NULL");
  if (!ckv_api::aligned(ws, 256)) return fail(CKV_UNSUPPORTED, "workspace must be 256-byte aligned");
  const int es = p->dtype == CKV_BF16 ? 2 : 4;
  char *w = static_cast<char *>(ws);
  ckv::DecArgs a{};
  a.q = static_cast<const char *>(q_dec);
  a.k = static_cast<const char *>(k);
  a.v = static_cast<const char *>(v);
  a.k_out = static_cast<const char *>(k_out);
  a.v_out = static_cast<const char *>(v_out);
  a.cu = p->cu_seqlens;
  a.part_ml = reinterpret_cast<float2 *>(w + pl.ml_off);
  a.part_o = reinterpret_cast<float *>(w + pl.o_off);
  a.a = reinterpret_cast<float *>(w + pl.a_off);
  a.k_st = p->k_stride_tok * es;
  a.k_sh = p->k_stride_head * es;
  a.v_st = p->v_stride_tok * es;
  a.v_sh = p->v_stride_head * es;
  a.Hq = p->n_q_heads;
  a.Hkv = p->n_kv_heads;
  a.G = p->n_q_heads / p->n_kv_heads;
  a.B = e->budget;
  a.n_chunks = pl.n_chunks;
  a.q_T = e->n_steps;
  const double scale = p->scale > 0.f ? (double)p->scale : 1.0 / std::sqrt((double)p->head_dim);
  a.c1 = (float)(scale * 1.4426950408889634);
  ckv::ProjArgs pa{};
  pa.w_o = static_cast<const char *>(w_o);
  pa.a = a.a;
  pa.part_ss = reinterpret_cast<float *>(w + pl.ss_off);
  pa.d_model = e->d_model;
  pa.HD = p->n_q_heads * p->head_dim;
  hipStream_t s = (hipStream_t)stream;
  // blocks of sequences x steps, sequences outermost: the sum runs over the
  // vectors (sequence, step) in that order
  bool first = true;
  for (int b0 = 0; b0 < p->batch; b0 += pl.BS) {
    for (int t0 = 0; t0 < e->n_steps; t0 += pl.TS) {
      a.b0 = b0;
      a.t0 = t0;
      a.batch = std::min(pl.BS, p->batch - b0);
      a.T = std::min(pl.TS, e->n_steps - t0);
      a.R = a.T * a.G;
      pa.NV = a.batch * a.T;
      const int rt = (a.R + 15) / 16;
      if (p->dtype == CKV_BF16) {
        if (p->head_dim == 64)
          ckv::launch_dec_t<__bf16, 64>(a, pa, rt, pl.n_wg, e->eps, first, err, s);
        else
          ckv::launch_dec_t<__bf16, 128>(a, pa, rt, pl.n_wg, e->eps, first, err, s);
      } else {
        if (p->head_dim == 64)
          ckv::launch_dec_t<float, 64>(a, pa, rt, pl.n_wg, e->eps, first, err, s);
        else
          ckv::launch_dec_t<float, 128>(a, pa, rt, pl.n_wg, e->eps, first, err, s);
      }
      first = false;
    }
  }
  const hipError_t he = hipGetLastError();
  if (he != hipSuccess)
    return fail(CKV_HIP_ERROR, "layer error launch failed: %s", hipGetErrorString(he));
  return ok();
}

}  // extern "C"
