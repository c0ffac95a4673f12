// Scoring kernels of the CompressKV eviction path (steps S1-S4) for gfx950:
// templates, instantiated for single-layer calls in score_kernels.hip and for
// the multi-layer entry point in score_layers.hip.
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
//                  in LDS, averages over the SRHs, and adds the scores to a
//                  2048-bin histogram of their top bits (first digit of the
//                  radix selection, S5).
//
// Rows of a KV group: SRH h (in head order) owns th = ceil(W/16) row tiles of
// 16 rows; row i < W of the tile set is window query i of that head, the
// padding rows have zero queries and are ignored.  A workgroup (8 waves)
// stages the group's window queries in LDS once; each wave keeps them in
// registers when they fit (up to 4 row tiles) and otherwise reads them from
// LDS per MFMA.  Each wave streams its key tiles through a two-deep pipeline
// of 2-tile groups (8 KB each): loads are unconditional (key index clamped
// into the sequence, extra tiles masked), so the compiler can wait for exactly
// the group being consumed while the next one is still in flight.
//
// ML (multi-layer): grid z runs over (layer, sequence) pairs, layer-major, and
// the layer's operands come from the table; otherwise from the arguments.
#pragma once

#include "score_common.h"

namespace ckv {

// ---------------------------------------------------------------------------
// S1+S2 partial statistics.  Grid (Hkv, ceil(max_chunks1 / cpw1), batch
// [x layers]), 64 * kStatsWaves threads; a workgroup covers cpw1 consecutive
// chunks of one (sequence, group) and writes one partial per chunk.  The
// groups of one key range are neighbours in launch order, so the workgroups in
// flight read whole token rows of K ([T, Hkv, D]) rather than 1/Hkv of each.
// MFMA operands: A = 16 keys, B = 16 window rows, so lane (quad, c) holds the
// logits of row c against keys 4*quad .. 4*quad+3 of the tile and keeps one
// running (ref, sum) pair per row tile.  Wave w handles the key tiles
// w, w + NW, w + 2 NW, ... of the workgroup's range; a chunk (chunk1 keys) is
// a whole number of 2-tile groups of every wave, so its partial is the same
// whichever workgroup size covers it.
// ---------------------------------------------------------------------------
constexpr int kStatsWaves = 4;

template <typename T, int D, int RTM, bool ML>
__global__ __launch_bounds__(64 * kStatsWaves) void stats_kernel(const ScoreArgs a) {
  constexpr int NW = kStatsWaves;
  constexpr int NS = Slices<T, D>::n, RQ = RegTiles<T, D, RTM>::v;
  constexpr int NT = 64 * NW;
  const int g = blockIdx.x;
  const int layer = ML ? (int)blockIdx.z / a.batch : 0;
  const int b = (int)blockIdx.z - layer * a.batch;
  const LayerView lv = layer_view<ML>(a, layer, g);
  const gptr<const char> kbase = lv.k;
  const int s0 = a.cu[b];
  const int L = a.cu[b + 1] - s0;
  const int chunk0 = (int)blockIdx.y * a.cpw1;
  if (chunk0 == 0) {   // the column-sum kernel accumulates this histogram afterwards
    int *h = a.hist + layer * a.hist_layer + ((int64_t)b * a.Hkv + g) * kHistBins;
    for (int i = threadIdx.x; i < kHistBins; i += NT) h[i] = 0;
  }
  const int c0 = chunk0 * a.chunk1;
  if (c0 >= L) return;                       // uniform for the whole workgroup
  const int n_chunks = min(a.cpw1, (L - c0 + a.chunk1 - 1) / a.chunk1);
  const int P = L - a.W;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int c = lane & 15, quad = lane >> 4;
  const int tid = threadIdx.x;
  const int rt_n = lv.nsrh * a.th;
  const int gpc = a.chunk1 / (16 * NW * kPair);   // 2-tile groups per wave and chunk (even)
  const int n_groups = gpc * n_chunks;
  // key row of this lane for tile index i of this wave, clamped into the range
  // (the pipeline's reads past the last tile hit the same cached row)
  const int k_last = min(L, c0 + n_chunks * a.chunk1) - 1;
  auto key_of = [&](int i) { return min(c0 + 16 * (wave + NW * i) + c, k_last); };
  float2 *parts = a.stats + layer * a.stats_layer +
                  ((int64_t)b * a.Hkv + g) * a.parts_stride * a.row_slots;

  __shared__ uint4 q_lds[RTM * 16 * QLayout<T, D>::STRIDE];
  __shared__ float2 part[NW][RTM * 16];

  // Query loads first, then the first two key groups; the queries are written
  // to LDS while the keys are still in flight.
  uint4 qv[QStage<T, D, RTM, NT>::n];
  q_load<T, D, RTM, NT>(a, lv, b, rt_n, qv);
  uint4 ka[kPair][NS], kb[kPair][NS];
#pragma unroll
  for (int p = 0; p < kPair; ++p) load_k_row<T, D>(a, kbase, s0, key_of(p), g, quad, ka[p]);
#pragma unroll
  for (int p = 0; p < kPair; ++p)
    load_k_row<T, D>(a, kbase, s0, key_of(kPair + p), g, quad, kb[p]);
  q_store<T, D, RTM, NT>(qv, q_lds);
  __syncthreads();
  uint4 qreg[RegTiles<T, D, RTM>::n][NS];
#pragma unroll
  for (int rt = 0; rt < RQ; ++rt)
#pragma unroll
    for (int s = 0; s < NS; ++s) qreg[rt][s] = q_frag<T, D>(q_lds, rt, s, c, quad);

  float ref[RTM], sum[RTM];
#pragma unroll
  for (int rt = 0; rt < RTM; ++rt) {
    ref[rt] = -INFINITY;
    sum[rt] = 0.f;
  }
  auto consume = [&](uint4 (&kf)[kPair][NS], int grp) {
#pragma unroll
    for (int p = 0; p < kPair; ++p) {
      const int base = c0 + 16 * (wave + NW * (kPair * grp + p));
      f32x4 acc[RTM];
#pragma unroll
      for (int rt = 0; rt < RTM; ++rt)
        if (rt < rt_n) acc[rt] = tile_logits<T, D, RTM, true>(kf[p], qreg, q_lds, rt, c, quad);
      stats_update<RTM>(a, acc, ref, sum, rt_n, base, L, P, c, quad);
    }
  };
  // The chunk's partial: merge the four quads (same row c, different keys),
  // then the waves in order, and start the next chunk from empty pairs.
  auto flush = [&](int chunk) {
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
    if (tid < rt_n * 16) {
      float r0 = part[0][tid].x, s_0 = part[0][tid].y;
#pragma unroll
      for (int w = 1; w < NW; ++w) merge_stats(r0, s_0, part[w][tid].x, part[w][tid].y);
      parts[(int64_t)chunk * a.row_slots + tid] = make_float2(r0, s_0);
    }
    __syncthreads();   // part is reused by the next chunk
#pragma unroll
    for (int rt = 0; rt < RTM; ++rt) {
      ref[rt] = -INFINITY;
      sum[rt] = 0.f;
    }
  };
  int chunk = chunk0;
  for (int grp = 0; grp < n_groups; grp += 2) {
    consume(ka, grp);
#pragma unroll
    for (int p = 0; p < kPair; ++p)
      load_k_row<T, D>(a, kbase, s0, key_of(kPair * (grp + 2) + p), g, quad, ka[p]);
    consume(kb, grp + 1);
#pragma unroll
    for (int p = 0; p < kPair; ++p)
      load_k_row<T, D>(a, kbase, s0, key_of(kPair * (grp + 3) + p), g, quad, kb[p]);
    if ((grp + 2) % gpc == 0) flush(chunk++);   // loads of the next chunk are in flight
  }
}

// ---------------------------------------------------------------------------
// S2+S3+S4.  Grid (Hkv, ceil(max_chunks2 / cpw2), batch [x layers]), 512
// threads; a workgroup covers cpw2 consecutive chunks of chunk2 keys.
// MFMA operands: A = 16 window rows, B = 16 keys, so lane (quad, c) holds
// rows 4*quad .. 4*quad+3 of the tile against key c.  The tiles of a chunk
// plus one halo tile on each side, e = -1 .. chunk2/16, go to the waves
// round-robin (chunk2 + 32 keys = 16 * kWaves * kPair * groups per chunk);
// the pipeline runs on across chunks, each chunk ending with its pooling.
// ---------------------------------------------------------------------------
template <typename T, int D, int RTM, bool ML>
__global__ __launch_bounds__(64 * kWaves) void colsum_kernel(const ScoreArgs a) {
  constexpr int NS = Slices<T, D>::n, RQ = RegTiles<T, D, RTM>::v;
  constexpr int NT = 64 * kWaves;
  constexpr int kMaxSrh = RTM;   // th >= 1
  const int g = blockIdx.x;
  const int layer = ML ? (int)blockIdx.z / a.batch : 0;
  const int b = (int)blockIdx.z - layer * a.batch;
  const LayerView lv = layer_view<ML>(a, layer, g);
  const gptr<const char> kbase = lv.k;
  const int s0 = a.cu[b];
  const int L = a.cu[b + 1] - s0;
  const int c0 = (int)blockIdx.y * a.cpw2 * a.chunk2;
  if (c0 >= L) return;
  const int c_end = min(L, c0 + a.cpw2 * a.chunk2);
  const int P = L - a.W;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int c = lane & 15, quad = lane >> 4;
  const int tid = threadIdx.x;
  const int nh = lv.nsrh;
  const int rt_n = nh * a.th;
  const gptr<float> out = lv.scores + (int64_t)g * a.T + s0;

  // Window positions of this range are always kept: +inf.
  for (int j = max(c0, P) + tid; j < c_end; j += NT) out[j] = INFINITY;
  if (c0 >= P) return;                        // no prefix key in this range
  // chunks of the range that hold prefix keys
  const int n_chunks = min(a.cpw2, (P - c0 + a.chunk2 - 1) / a.chunk2);
  const int gpc = (a.chunk2 + 32) / (16 * kWaves * kPair);   // 2-tile groups per wave and chunk
  const int n_groups = gpc * n_chunks;
  // chunk, tile index e in the chunk and key row of this lane for the i-th
  // tile of this wave (clamped into the chunk and its halo)
  auto key_of = [&](int i) {
    const int grp = i / kPair;
    const int ch = grp / gpc;
    const int e = -1 + wave + kWaves * (i - ch * gpc * kPair);
    const int cc0 = c0 + ch * a.chunk2;
    const int k_first = max(cc0 - 16, 0), k_last = min(cc0 + a.chunk2 + 16, L) - 1;
    return min(max(cc0 + 16 * e + c, k_first), k_last);
  };

  __shared__ uint4 q_lds[RTM * 16 * QLayout<T, D>::STRIDE];
  __shared__ float bias_s[RTM * 16];
  __shared__ float cs[kMaxSrh][kMaxChunk2 + 32];
  __shared__ int hist_s[kHistBins];
  uint4 qv[QStage<T, D, RTM, NT>::n];
  q_load<T, D, RTM, NT>(a, lv, b, rt_n, qv);
  uint4 ka[kPair][NS], kb[kPair][NS];
#pragma unroll
  for (int p = 0; p < kPair; ++p) load_k_row<T, D>(a, kbase, s0, key_of(p), g, quad, ka[p]);
#pragma unroll
  for (int p = 0; p < kPair; ++p)
    load_k_row<T, D>(a, kbase, s0, key_of(kPair + p), g, quad, kb[p]);
  q_store<T, D, RTM, NT>(qv, q_lds);
  for (int i = tid; i < kHistBins; i += NT) hist_s[i] = 0;

  // Row normalisers bias = ref + log2(sum), merged over every chunk of the
  // statistics pass.
  merge_row_bias<NT>(a,
                     a.stats + layer * a.stats_layer +
                         ((int64_t)b * a.Hkv + g) * a.parts_stride * a.row_slots,
                     a.row_slots, (L + a.chunk1 - 1) / a.chunk1, rt_n * 16, RTM * 16, bias_s);
  __syncthreads();
  uint4 qreg[RegTiles<T, D, RTM>::n][NS];
#pragma unroll
  for (int rt = 0; rt < RQ; ++rt)
#pragma unroll
    for (int s = 0; s < NS; ++s) qreg[rt][s] = q_frag<T, D>(q_lds, rt, s, c, quad);
  float bias[RTM][4];
#pragma unroll
  for (int rt = 0; rt < RTM; ++rt)
#pragma unroll
    for (int r = 0; r < 4; ++r) bias[rt][r] = bias_s[rt * 16 + 4 * quad + r];

  // Column sums of a chunk plus one 16-key halo tile on each side:
  // cs[h][16 + x] holds the window sum of SRH h at key cc0 + x.
  auto consume = [&](uint4 (&kf)[kPair][NS], int grp) {
    const int ch = grp / gpc;
    const int cc0 = c0 + ch * a.chunk2;
    const int p_end = min(cc0 + a.chunk2, P);
    const int ntiles = (p_end - cc0 + 15) >> 4;                       // tiles e = 0 .. ntiles-1
    const int e_lo = (cc0 > 0) ? -1 : 0;                              // left halo tile
    const int e_hi = (cc0 + 16 * ntiles < P) ? ntiles : ntiles - 1;   // right halo tile
#pragma unroll
    for (int p = 0; p < kPair; ++p) {
      const int e = -1 + wave + kWaves * (kPair * (grp - ch * gpc) + p);
      tile_window_sums<T, D, RTM, kMaxChunk2 + 32>(a, kf[p], qreg, q_lds, bias, rt_n, e,
                                                   e >= e_lo && e <= e_hi, c, quad, cs);
    }
  };
  // Pooling of a finished chunk (S4); cs is rewritten by the next chunk only
  // after every thread has pooled.
  auto pool = [&](int ch) {
    const int cc0 = c0 + ch * a.chunk2;
    __syncthreads();
    pool_scores<NT, kMaxChunk2 + 32>(a, cs, nh, cc0, min(cc0 + a.chunk2, P), P, out, hist_s);
    __syncthreads();
  };
  for (int grp = 0; grp < n_groups; grp += 2) {
    consume(ka, grp);
#pragma unroll
    for (int p = 0; p < kPair; ++p)
      load_k_row<T, D>(a, kbase, s0, key_of(kPair * (grp + 2) + p), g, quad, ka[p]);
    consume(kb, grp + 1);
#pragma unroll
    for (int p = 0; p < kPair; ++p)
      load_k_row<T, D>(a, kbase, s0, key_of(kPair * (grp + 3) + p), g, quad, kb[p]);
    if ((grp + 2) % gpc == 0) pool(grp / gpc);   // loads of the next chunk are in flight
  }
  flush_hist<NT>(hist_s, a.hist + layer * a.hist_layer + ((int64_t)b * a.Hkv + g) * kHistBins);
}

// ---------------------------------------------------------------------------
// Host-side launcher template; grid z = batch * n_layers (n_layers = 1 unless ML).
// ---------------------------------------------------------------------------
template <typename T, int D, int RTM, bool ML>
static hipError_t launch_score_t(const ScoreArgs &a, int nz, hipStream_t stream) {
  const int y1 = (a.max_chunks1 + a.cpw1 - 1) / a.cpw1;
  const int y2 = (a.max_chunks2 + a.cpw2 - 1) / a.cpw2;
  hipLaunchKernelGGL((stats_kernel<T, D, RTM, ML>), dim3(a.Hkv, y1, nz), dim3(64 * kStatsWaves),
                     0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((colsum_kernel<T, D, RTM, ML>), dim3(a.Hkv, y2, nz), dim3(64 * kWaves), 0,
                     stream, a);
  return hipGetLastError();
}

template <typename T, int D, bool ML>
static hipError_t launch_score_d(const ScoreArgs &a, int rt_max, int nz, hipStream_t stream) {
  switch (rt_max) {
    case 1: return launch_score_t<T, D, 1, ML>(a, nz, stream);
    case 2: return launch_score_t<T, D, 2, ML>(a, nz, stream);
    case 3: return launch_score_t<T, D, 3, ML>(a, nz, stream);
    case 4: return launch_score_t<T, D, 4, ML>(a, nz, stream);
    case 5:
    case 6: return launch_score_t<T, D, 6, ML>(a, nz, stream);
    case 7:
    case 8: return launch_score_t<T, D, 8, ML>(a, nz, stream);
    default: return launch_score_t<T, D, 12, ML>(a, nz, stream);
  }
}

template <bool ML>
static hipError_t launch_score_any(const ScoreArgs &a, int dtype_bf16, int head_dim, int rt_max,
                                   int nz, hipStream_t stream) {
  if (dtype_bf16) {
    return head_dim == 64 ? launch_score_d<__bf16, 64, ML>(a, rt_max, nz, stream)
                          : launch_score_d<__bf16, 128, ML>(a, rt_max, nz, stream);
  }
  return head_dim == 64 ? launch_score_d<float, 64, ML>(a, rt_max, nz, stream)
                        : launch_score_d<float, 128, ML>(a, rt_max, nz, stream);
}

}  // namespace ckv
