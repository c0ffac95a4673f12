// Eviction error of a layer (section 3.4, equations 2-4): over decoding steps,
// ||W_O (A_full - A_comp)||_F / (||W_O A_full||_F + eps), where A is the
// attention of the step's queries over the full KV cache or over the compact
// cache that the eviction path wrote.
//
//   dec_attn_kernel     split-K attention of every (sequence, group, cache):
//                       the group's rows (decoding step x query head of the
//                       group) against one 512-key chunk, QK^T on MFMA, online
//                       softmax in LDS, P.V on the VALU; partial (max, sum, O)
//   dec_combine_kernel  merges the chunks of every row into A (fp32)
//   dec_proj_kernel     y = W_O x for x = A_full and A_full - A_comp, 64 rows of
//                       W_O per workgroup; per-workgroup sums of y^2
//   dec_error_kernel    the per-step norms, their ratios and the layer sum
//
// Every reduction runs in a fixed order, so the result is deterministic.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>

#include "../../include/compresskv_offline.h"
#include "api_common.h"
#include "score_common.h"

namespace ckv {

constexpr int kDecChunk = 512;   // keys per attention workgroup
constexpr int kDecSub = 128;     // keys per softmax step inside it (8 tiles)
constexpr int kProjRows = 64;    // W_O rows per projection workgroup
constexpr int kMaxDecRows = 64;  // decoding steps x query heads per group
constexpr int kMaxVectors = 32;  // sequences x decoding steps

struct DecArgs {
  const char *q;                 // [batch][T][Hq][D]
  const char *k, *v;             // full caches, byte strides below
  const char *k_out, *v_out;     // compact caches [batch][Hkv][B][D]
  const int32_t *cu;
  float2 *part_ml;               // [2][batch][Hkv][n_chunks][64] (max, sum), log2 domain
  float *part_o;                 // [2][batch][Hkv][n_chunks][64][D]
  float *a;                      // [2][batch][T][Hq][D]
  int64_t k_st, k_sh, v_st, v_sh;
  int T, Hq, Hkv, G, B, batch, R, n_chunks;
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
// queries.  Thread (rb, db) of the P.V step owns rows rb*RPT .. +RPT and
// columns 4*db .. 4*db+3.
template <typename T, int D, int RT>
__global__ __launch_bounds__(256) void dec_attn_kernel(const DecArgs a) {
  constexpr int NS = Slices<T, D>::n, U4 = QLayout<T, D>::U4, STRIDE = QLayout<T, D>::STRIDE;
  constexpr int RP = RT * 16;                  // rows with padding
  constexpr int DB = D / 4, RB = 256 / DB;     // column and row blocks of the P.V step
  constexpr int RPT = RP / RB;                 // rows per thread there (>= 1)
  constexpr int ZS = kDecSub + 1;              // padded row of the logits buffer
  static_assert(RP % RB == 0, "row blocks");
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int c = lane & 15, quad = lane >> 4;
  const int g = blockIdx.y, b = (int)blockIdx.z >> 1, cache = (int)blockIdx.z & 1;
  const DecCache cc = dec_cache<T, D>(a, cache, b, g);
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
      val = load16(to_global(a.q) + (((int64_t)b * a.T + t) * a.Hq + h) * (D * (int64_t)sizeof(T)) +
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

  const int rb = tid / DB, db = tid - rb * DB;
  float acc[RPT][4];
#pragma unroll
  for (int i = 0; i < RPT; ++i)
#pragma unroll
    for (int d = 0; d < 4; ++d) acc[i][d] = 0.f;

  for (int k0 = c0; k0 < c_end; k0 += kDecSub) {
    // S: logits of the step's 8 key tiles (2 per wave), scaled to log2 units
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int e = wave + 4 * i;
      const int key = min(k0 + 16 * e + c, cc.n_keys - 1);
      uint4 kf[NS];
      const gptr<const char> p = to_global(cc.kb) + key * cc.k_row + 16 * quad;
#pragma unroll
      for (int s = 0; s < NS; ++s) kf[s] = load16(p + 64 * s);
      f32x4 lg[RT];
      tile_logits_all<T, D, RT, true>(kf, qreg, q_lds, c, quad, lg);
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int j = 16 * e + 4 * quad + r;
          zs[(rt * 16 + c) * ZS + j] = (k0 + j < c_end) ? lg[rt][r] * a.c1 : -INFINITY;
        }
    }
    // V rows of the step
    {
      constexpr int V4 = D * (int)sizeof(T) / 16;   // 16-byte units per row
      for (int i = tid; i < kDecSub * V4; i += 256) {
        const int j = i / V4, u = i - j * V4;
        const int key = min(k0 + j, cc.n_keys - 1);
        const uint4 val = load16(to_global(cc.vb) + key * cc.v_row + 16 * u);
        vs4[i] = val;
      }
    }
    __syncthreads();
    // online softmax: four threads per row, 32 keys each
    {
      const int r = tid >> 2, part = tid & 3;
      if (r < RP) {
        float* zr = zs + r * ZS + 32 * part;
        float mx = -INFINITY;
        for (int j = 0; j < 32; ++j) mx = fmaxf(mx, zr[j]);
        mx = fmaxf(mx, __shfl_xor(mx, 1));
        mx = fmaxf(mx, __shfl_xor(mx, 2));
        const float m_old = m_s[r];
        const float m_new = fmaxf(m_old, mx);
        // a row with no visible key yet keeps zero weight
        const float alpha = (m_new == -INFINITY) ? 1.f : fast_exp2(m_old - m_new);
        float sm = 0.f;
        for (int j = 0; j < 32; ++j) {
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
    // O = alpha * O + P.V
#pragma unroll
    for (int i = 0; i < RPT; ++i) {
      const int r = rb * RPT + i;
      const float al = alpha_s[r];
#pragma unroll
      for (int d = 0; d < 4; ++d) acc[i][d] *= al;
    }
    const int nk = min(kDecSub, c_end - k0);
    for (int j = 0; j < nk; ++j) {
      float vv[4];
#pragma unroll
      for (int d = 0; d < 4; ++d) vv[d] = (float)vs[j * D + 4 * db + d];
#pragma unroll
      for (int i = 0; i < RPT; ++i) {
        const float p = zs[(rb * RPT + i) * ZS + j];
#pragma unroll
        for (int d = 0; d < 4; ++d) acc[i][d] = __builtin_fmaf(p, vv[d], acc[i][d]);
      }
    }
    __syncthreads();   // zs and vs are rewritten by the next step
  }
  // partials of this chunk
  const int64_t slot = (((int64_t)cache * a.batch + b) * a.Hkv + g) * a.n_chunks + blockIdx.x;
  if (tid < a.R) a.part_ml[slot * kMaxDecRows + tid] = make_float2(m_s[tid], l_s[tid]);
#pragma unroll
  for (int i = 0; i < RPT; ++i) {
    const int r = rb * RPT + i;
    if (r < a.R) {
      float *o = a.part_o + (slot * kMaxDecRows + r) * D + 4 * db;
#pragma unroll
      for (int d = 0; d < 4; ++d) o[d] = acc[i][d];
    }
  }
}

// Grid (Hkv, batch * 2), 256 threads: A of every row of the group from its
// chunks, in chunk order.
template <int D>
__global__ __launch_bounds__(256) void dec_combine_kernel(const DecArgs a) {
  const int g = blockIdx.x, b = (int)blockIdx.y >> 1, cache = (int)blockIdx.y & 1;
  const int L = a.cu[b + 1] - a.cu[b];
  const int n_keys = cache == 0 ? L : min(L, a.B);
  const int nch = (n_keys + kDecChunk - 1) / kDecChunk;
  const int64_t slot0 = (((int64_t)cache * a.batch + b) * a.Hkv + g) * a.n_chunks;
  for (int i = threadIdx.x; i < a.R * D; i += 256) {
    const int r = i / D, d = i - r * D;
    float M = -INFINITY;
    for (int ch = 0; ch < nch; ++ch) M = fmaxf(M, a.part_ml[(slot0 + ch) * kMaxDecRows + r].x);
    float lsum = 0.f, o = 0.f;
    for (int ch = 0; ch < nch; ++ch) {
      const float2 ml = a.part_ml[(slot0 + ch) * kMaxDecRows + r];
      const float w = fast_exp2(ml.x - M);
      lsum += ml.y * w;
      o += a.part_o[((slot0 + ch) * kMaxDecRows + r) * D + d] * w;
    }
    const int t = r / a.G, h = g * a.G + (r - t * a.G);
    a.a[((((int64_t)cache * a.batch + b) * a.T + t) * a.Hq + h) * D + d] = o / lsum;
  }
}

struct ProjArgs {
  const char *w_o;          // [d_model][HD], dtype T
  const float *a;           // [2][NV][HD]: A_full, A_comp
  float *part_ss;           // [n_wg][2][NV]: sums of y_full^2, y_diff^2 over the workgroup's rows
  int d_model, HD, NV;
};

// Grid (ceil(d_model / 64)), 256 threads: thread (quarter, row) accumulates
// row o's dot products with every vector over a quarter of HD; the quarters
// are added in order, then the squares over the workgroup's rows.
template <typename T>
__global__ __launch_bounds__(256) void dec_proj_kernel(const ProjArgs p) {
  constexpr int KC = 256;   // columns staged per step
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int o = (int)blockIdx.x * kProjRows + lane;
  __shared__ float xs[2][kMaxVectors][KC];
  __shared__ float ys[4][kProjRows][2 * kMaxVectors + 1];
  float sf[kMaxVectors], sd[kMaxVectors];
#pragma unroll
  for (int n = 0; n < kMaxVectors; ++n) sf[n] = sd[n] = 0.f;
  const int quarter = KC / 4;
  for (int k0 = 0; k0 < p.HD; k0 += KC) {
    __syncthreads();
    for (int i = tid; i < p.NV * KC; i += 256) {
      const int n = i / KC, k = i - n * KC;
      const float f = p.a[(int64_t)n * p.HD + k0 + k];
      const float cmp = p.a[((int64_t)p.NV + n) * p.HD + k0 + k];
      xs[0][n][k] = f;
      xs[1][n][k] = f - cmp;
    }
    __syncthreads();
    if (o < p.d_model) {
      const T *wr = reinterpret_cast<const T *>(p.w_o) + (int64_t)o * p.HD + k0 + wave * quarter;
      for (int k = 0; k < quarter; ++k) {
        const float w = (float)wr[k];
        const int kk = wave * quarter + k;
#pragma unroll
        for (int n = 0; n < kMaxVectors; ++n) {
          if (n < p.NV) {
            sf[n] = __builtin_fmaf(w, xs[0][n][kk], sf[n]);
            sd[n] = __builtin_fmaf(w, xs[1][n][kk], sd[n]);
          }
        }
      }
    }
  }
#pragma unroll
  for (int n = 0; n < kMaxVectors; ++n) {
    ys[wave][lane][n] = sf[n];
    ys[wave][lane][kMaxVectors + n] = sd[n];
  }
  __syncthreads();
  // thread j < 2 NV: squares of the workgroup's rows in row order
  if (tid < 2 * p.NV) {
    const int col = tid < p.NV ? tid : kMaxVectors + (tid - p.NV);
    float ss = 0.f;
    for (int r = 0; r < kProjRows; ++r) {
      if ((int)blockIdx.x * kProjRows + r >= p.d_model) break;
      const float y = ((ys[0][r][col] + ys[1][r][col]) + ys[2][r][col]) + ys[3][r][col];
      ss = __builtin_fmaf(y, y, ss);
    }
    p.part_ss[((int64_t)blockIdx.x * 2 + (tid < p.NV ? 0 : 1)) * kMaxVectors +
              (tid < p.NV ? tid : tid - p.NV)] = ss;
  }
}

// One thread: per vector the norms over all workgroups (in order), the ratio,
// and the sum over vectors.
__global__ void dec_error_kernel(const float *part_ss, int n_wg, int NV, float eps, float *err) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  float e = 0.f;
  for (int n = 0; n < NV; ++n) {
    float sf = 0.f, sd = 0.f;
    for (int w = 0; w < n_wg; ++w) {
      sf += part_ss[((int64_t)w * 2 + 0) * kMaxVectors + n];
      sd += part_ss[((int64_t)w * 2 + 1) * kMaxVectors + n];
    }
    e += sqrtf(sd) / (sqrtf(sf) + eps);
  }
  err[0] = e;
}

template <typename T, int D>
static void launch_dec_t(const DecArgs &a, const ProjArgs &pa, int rt, int n_wg, float eps,
                         float *err, hipStream_t s) {
  const dim3 g1(a.n_chunks, a.Hkv, a.batch * 2);
  switch (rt) {
    case 1: hipLaunchKernelGGL((dec_attn_kernel<T, D, 1>), g1, dim3(256), 0, s, a); break;
    case 2: hipLaunchKernelGGL((dec_attn_kernel<T, D, 2>), g1, dim3(256), 0, s, a); break;
    case 3: hipLaunchKernelGGL((dec_attn_kernel<T, D, 3>), g1, dim3(256), 0, s, a); break;
    default: hipLaunchKernelGGL((dec_attn_kernel<T, D, 4>), g1, dim3(256), 0, s, a); break;
  }
  hipLaunchKernelGGL((dec_combine_kernel<D>), dim3(a.Hkv, a.batch * 2), dim3(256), 0, s, a);
  hipLaunchKernelGGL((dec_proj_kernel<T>), dim3(n_wg), dim3(256), 0, s, pa);
  hipLaunchKernelGGL(dec_error_kernel, dim3(1), dim3(64), 0, s, pa.part_ss, n_wg, pa.NV, eps,
                     err);
}

}  // namespace ckv

namespace {

using ckv_api::fail;
using ckv_api::ok;

struct DecPlan {
  int R = 0, rt = 0, n_chunks = 0, n_wg = 0, NV = 0, lmax = 0;
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
  pl.R = e->n_steps * G;
  if (pl.R > ckv::kMaxDecRows)
    return fail(CKV_UNSUPPORTED, "n_steps * (n_q_heads / n_kv_heads) must be <= %d",
                ckv::kMaxDecRows);
  pl.NV = p->batch * e->n_steps;
  if (pl.NV > ckv::kMaxVectors)
    return fail(CKV_UNSUPPORTED, "batch * n_steps must be <= %d", ckv::kMaxVectors);
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
  const size_t slots = (size_t)2 * p->batch * p->n_kv_heads * pl.n_chunks * ckv::kMaxDecRows;
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
  a.T = e->n_steps;
  a.Hq = p->n_q_heads;
  a.Hkv = p->n_kv_heads;
  a.G = p->n_q_heads / p->n_kv_heads;
  a.B = e->budget;
  a.batch = p->batch;
  a.R = pl.R;
  a.n_chunks = pl.n_chunks;
  const double scale = p->scale > 0.f ? (double)p->scale : 1.0 / std::sqrt((double)p->head_dim);
  a.c1 = (float)(scale * 1.4426950408889634);
  ckv::ProjArgs pa{};
  pa.w_o = static_cast<const char *>(w_o);
  pa.a = a.a;
  pa.part_ss = reinterpret_cast<float *>(w + pl.ss_off);
  pa.d_model = e->d_model;
  pa.HD = p->n_q_heads * p->head_dim;
  pa.NV = pl.NV;
  hipStream_t s = (hipStream_t)stream;
  if (p->dtype == CKV_BF16) {
    if (p->head_dim == 64)
      ckv::launch_dec_t<__bf16, 64>(a, pa, pl.rt, pl.n_wg, e->eps, err, s);
    else
      ckv::launch_dec_t<__bf16, 128>(a, pa, pl.rt, pl.n_wg, e->eps, err, s);
  } else {
    if (p->head_dim == 64)
      ckv::launch_dec_t<float, 64>(a, pa, pl.rt, pl.n_wg, e->eps, err, s);
    else
      ckv::launch_dec_t<float, 128>(a, pa, pl.rt, pl.n_wg, e->eps, err, s);
  }
  const hipError_t he = hipGetLastError();
  if (he != hipSuccess)
    return fail(CKV_HIP_ERROR, "layer error launch failed: %s", hipGetErrorString(he));
  return ok();
}

}  // extern "C"
