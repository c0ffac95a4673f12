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

// One wave per head; a workgroup of 4 waves covers 4 consecutive heads.  Per
// (sample, step) the wave tests whether the generated token is one of the
// span's tokens and, if so, sums the head's weights over the span (lanes over
// positions, then a fixed butterfly); the step sums accumulate in fp64.
__global__ __launch_bounds__(256) void srh_score_kernel(const SrhArgs a) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int h = blockIdx.x * 4 + wave;
  if (h >= a.H) return;   // whole waves; the kernel has no barrier
  double acc = 0.0;
  for (int s = 0; s < a.S; ++s) {
    const int a0 = a.spans[2 * s], n = a.spans[2 * s + 1];
    const int32_t *span_tok = a.ctx + (int64_t)s * a.L + a0;
    for (int t = 0; t < a.N; ++t) {
      const int32_t y = a.gen[(int64_t)s * a.N + t];
      bool hit = false;
      for (int j = lane; j < n; j += 64) hit |= (span_tok[j] == y);
      if (!__any(hit)) continue;   // uniform over the wave
      const float *row = a.attn + (((int64_t)s * a.N + t) * a.H + h) * (int64_t)a.L + a0;
      float v = 0.f;
      for (int j = lane; j < n; j += 64) v += row[j];
#pragma unroll
      for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
      acc += (double)v;
    }
  }
  if (lane == 0) a.scores[h] = (float)acc;
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
  hipLaunchKernelGGL(ckv::srh_score_kernel, dim3((p->n_heads + 3) / 4), dim3(256), 0,
                     (hipStream_t)stream, a);
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
