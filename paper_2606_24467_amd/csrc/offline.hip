// Offline analyses of CompressKV (include/compresskv_offline.h): the SRH
// score of every head (section 3.2, equation 1), each layer's SRH set
// (section 3.3) and the layer budgets from the layers' eviction errors
// (section 3.4; the errors themselves are computed in decode_error.hip).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <vector>

#include "../../include/compresskv_offline.h"
#include "api_common.h"

namespace ckv {

struct SrhArgs {
  const float *attn;
  const int32_t *gen, *ctx, *spans;
  float *scores;
  int32_t S, N, H, L;
};

constexpr int kSrhHeads = 4;        // heads per workgroup
constexpr int kSrhSplit = 4;        // waves per head
constexpr int kSrhBatch = 8;        // answer steps whose span loads a wave issues together
constexpr int kSrhPairs = 2048;     // (sample, step) pairs tested per pass

// A workgroup of 16 waves covers 4 consecutive heads.  Per block of (sample,
// step) pairs it first records in LDS whether each step generated one of its
// span's tokens (one thread per pair, looping over the span); the four
// waves of a head then take every fourth answer step of the block, load
// kSrhBatch spans together, sum each over the span (lanes over positions,
// then a fixed butterfly) and accumulate the step sums in fp64 in step
// order.  The four waves' totals are added in wave order, so the result does
// not depend on scheduling.
__global__ __launch_bounds__(64 * kSrhHeads * kSrhSplit) void srh_score_kernel(const SrhArgs a) {
  constexpr int NW = kSrhHeads * kSrhSplit;
  __shared__ unsigned char hit_s[kSrhPairs];
  __shared__ double part_s[NW];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int h = blockIdx.x * kSrhHeads + wave / kSrhSplit, sub = wave % kSrhSplit;
  const int SN = a.S * a.N;
  double acc = 0.0;
  for (int p0 = 0; p0 < SN; p0 += kSrhPairs) {
    const int np = min(kSrhPairs, SN - p0);
    for (int q = (int)threadIdx.x; q < np; q += 64 * NW) {
      const int p = p0 + q, s = p / a.N;
      const int a0 = a.spans[2 * s], n = a.spans[2 * s + 1];
      const int32_t y = a.gen[p];
      const int32_t *tok = a.ctx + (int64_t)s * a.L + a0;
      bool hit = false;
      for (int j = 0; j < n; ++j) hit |= (tok[j] == y);
      hit_s[q] = hit ? 1 : 0;
    }
    __syncthreads();
    if (h < a.H) {
      int q = sub;
      for (;;) {
        // the wave's next kSrhBatch answer steps of the block (uniform)
        int qb[kSrhBatch], nb = 0;
        while (nb < kSrhBatch && q < np) {
          if (hit_s[q]) qb[nb++] = q;
          q += kSrhSplit;
        }
        if (nb == 0) break;
        const float *row[kSrhBatch];
        int len[kSrhBatch], nmax = 0;
#pragma unroll
        for (int b = 0; b < kSrhBatch; ++b) {
          const int p = p0 + (b < nb ? qb[b] : qb[0]), s = p / a.N;
          const int a0 = a.spans[2 * s];
          len[b] = b < nb ? a.spans[2 * s + 1] : 0;
          row[b] = a.attn + ((int64_t)p * a.H + h) * (int64_t)a.L + a0;
          nmax = max(nmax, len[b]);
        }
        float v[kSrhBatch];
#pragma unroll
        for (int b = 0; b < kSrhBatch; ++b) v[b] = 0.f;
        for (int j = lane; j < nmax; j += 64) {
          float x[kSrhBatch];
#pragma unroll
          for (int b = 0; b < kSrhBatch; ++b) x[b] = (j < len[b]) ? row[b][j] : 0.f;
#pragma unroll
          for (int b = 0; b < kSrhBatch; ++b) v[b] += x[b];
        }
#pragma unroll
        for (int b = 0; b < kSrhBatch; ++b) {
#pragma unroll
          for (int o = 32; o >= 1; o >>= 1) v[b] += __shfl_xor(v[b], o);
          if (b < nb) acc += (double)v[b];
        }
      }
    }
    __syncthreads();   // hit_s is rewritten by the next block
  }
  if (lane == 0) part_s[wave] = acc;
  __syncthreads();
  if (sub == 0 && lane == 0 && h < a.H) {
    double t = 0.0;
#pragma unroll
    for (int w = 0; w < kSrhSplit; ++w) t += part_s[wave + w];
    a.scores[h] = (float)t;
  }
}

// One workgroup per layer, one thread per head: a head's rank is the number of
// heads with a higher score or an equal score and a lower index.
__global__ __launch_bounds__(1024) void select_srh_kernel(const float *scores, int hp, int top_k,
                                                          uint8_t *mask) {
  const int l = blockIdx.x, h = threadIdx.x;
  if (h >= hp) return;
  const float *sc = scores + (int64_t)l * hp;
  const float me = sc[h];
  int rank = 0;
  for (int o = 0; o < hp; ++o) {
    const float x = sc[o];
    rank += (x > me) || (x == me && o < h);
  }
  mask[(int64_t)l * hp + h] = rank < top_k ? 1 : 0;
}

}  // namespace ckv

using ckv_api::fail;
using ckv_api::ok;

extern "C" {

int compresskv_srh_scores(const ckv_srh_problem *p, const float *attn, const int32_t *gen_tokens,
                          const int32_t *ctx_tokens, const int32_t *spans, float *scores,
                          void *stream) {
  if (!p) return fail(CKV_INVALID_ARGUMENT, "problem is NULL");
  if (p->n_samples < 1 || p->n_steps < 1 || p->n_heads < 1 || p->ctx_len < 1)
    return fail(CKV_INVALID_ARGUMENT, "n_samples, n_steps, n_heads and ctx_len must be >= 1");
  if (!p->spans_host) return fail(CKV_INVALID_ARGUMENT, "spans_host is NULL");
  for (int s = 0; s < p->n_samples; ++s) {
    const int a0 = p->spans_host[2 * s], n = p->spans_host[2 * s + 1];
    if (a0 < 0 || n < 1 || (int64_t)a0 + n > p->ctx_len)
      return fail(CKV_INVALID_ARGUMENT, "sample %d: span (%d, %d) outside [0, %d)", s, a0, n,
                  p->ctx_len);
  }
  const void *ptrs[] = {attn, gen_tokens, ctx_tokens, spans, scores};
  const char *names[] = {"attn", "gen_tokens", "ctx_tokens", "spans", "scores"};
  for (int i = 0; i < 5; ++i) {
    if (!ptrs[i]) return fail(CKV_INVALID_ARGUMENT, "%s is NULL", names[i]);
    if (!ckv_api::aligned(ptrs[i], 4))
      return fail(CKV_UNSUPPORTED, "%s must be 4-byte aligned", names[i]);
  }
  ckv::SrhArgs a{attn, gen_tokens, ctx_tokens, spans, scores,
                 p->n_samples, p->n_steps, p->n_heads, p->ctx_len};
  hipLaunchKernelGGL(ckv::srh_score_kernel, dim3((p->n_heads + ckv::kSrhHeads - 1) / ckv::kSrhHeads),
                     dim3(64 * ckv::kSrhHeads * ckv::kSrhSplit), 0, (hipStream_t)stream, a);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess)
    return fail(CKV_HIP_ERROR, "srh score launch failed: %s", hipGetErrorString(e));
  return ok();
}

int compresskv_select_srh(int32_t n_layers, int32_t heads_per_layer, const float *scores,
                          int32_t top_k, uint8_t *srh_mask, void *stream) {
  if (n_layers < 1 || n_layers > 65535)
    return fail(CKV_INVALID_ARGUMENT, "n_layers must be in [1, 65535] (got %d)", n_layers);
  if (heads_per_layer < 1 || heads_per_layer > 1024)
    return fail(CKV_UNSUPPORTED, "heads_per_layer must be in [1, 1024] (got %d)",
                heads_per_layer);
  if (top_k < 1 || top_k > heads_per_layer)
    return fail(CKV_INVALID_ARGUMENT, "top_k must be in [1, heads_per_layer] (got %d)", top_k);
  if (!scores || !srh_mask) return fail(CKV_INVALID_ARGUMENT, "scores and srh_mask are required");
  if (!ckv_api::aligned(scores, 4)) return fail(CKV_UNSUPPORTED, "scores must be 4-byte aligned");
  hipLaunchKernelGGL(ckv::select_srh_kernel, dim3(n_layers), dim3(heads_per_layer), 0,
                     (hipStream_t)stream, scores, (int)heads_per_layer, (int)top_k, srh_mask);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess)
    return fail(CKV_HIP_ERROR, "select srh launch failed: %s", hipGetErrorString(e));
  return ok();
}

int compresskv_allocate_budgets(int32_t n_layers, const float *errors_host, int64_t total,
                                int32_t min_budget, int32_t max_budget, int32_t *budgets_host) {
  if (n_layers < 1) return fail(CKV_INVALID_ARGUMENT, "n_layers must be >= 1 (got %d)", n_layers);
  if (!errors_host || !budgets_host)
    return fail(CKV_INVALID_ARGUMENT, "errors_host and budgets_host are required");
  if (min_budget < 1 || max_budget < min_budget)
    return fail(CKV_INVALID_ARGUMENT, "need 1 <= min_budget <= max_budget");
  const int n = n_layers;
  if (total < (int64_t)n * min_budget || total > (int64_t)n * max_budget)
    return fail(CKV_INVALID_ARGUMENT, "total must lie in [n_layers * min, n_layers * max]");
  double esum = 0.0;
  for (int i = 0; i < n; ++i) {
    const float e = errors_host[i];
    if (!std::isfinite(e) || e < 0.f)
      return fail(CKV_INVALID_ARGUMENT, "layer %d: error must be finite and >= 0", i);
    esum += e;
  }
  // normalised errors (a layer set of all-zero errors shares evenly)
  std::vector<double> w(n), share(n, 0.0);
  for (int i = 0; i < n; ++i) w[i] = esum > 0.0 ? (double)errors_host[i] / esum : 0.0;
  std::vector<char> capped(n, 0);
  for (;;) {
    int n_free = 0;
    double wsum = 0.0;
    for (int i = 0; i < n; ++i)
      if (!capped[i]) {
        ++n_free;
        wsum += w[i];
      }
    const double rest =
        (double)(total - (int64_t)(n - n_free) * max_budget - (int64_t)n_free * min_budget);
    bool over = false;
    for (int i = 0; i < n; ++i) {
      if (capped[i]) continue;
      share[i] = wsum > 0.0 ? rest * w[i] / wsum : rest / n_free;
      over |= (min_budget + share[i] > max_budget);
    }
    if (!over) break;
    for (int i = 0; i < n; ++i)
      if (!capped[i] && min_budget + share[i] > max_budget) capped[i] = 1;
  }
  int64_t used = 0;
  std::vector<int> order;
  for (int i = 0; i < n; ++i) {
    if (capped[i]) {
      budgets_host[i] = max_budget;
    } else {
      budgets_host[i] = min_budget + (int32_t)std::floor(share[i]);
      order.push_back(i);
    }
    used += budgets_host[i];
  }
  // the units left by rounding down: largest fractional parts first
  std::stable_sort(order.begin(), order.end(), [&](int x, int y) {
    return share[x] - std::floor(share[x]) > share[y] - std::floor(share[y]);
  });
  for (int64_t left = total - used, j = 0; left > 0 && j < (int64_t)order.size(); --left, ++j)
    budgets_host[order[j]] += 1;
  return ok();
}

}  // extern "C"
