// Scoring kernels of the CompressKV eviction path (steps S1-S4) for gfx950:
// templates, instantiated for single-layer calls in score_kernels.hip and for
// the multi-layer entry point in score_layers.hip.
//
// The window softmax (section 3.3, SnapKV-style window of section 4) needs each
// window row's statistics over the whole sequence before any column can be
// normalised, so scoring makes two passes over K, either as two kernels or as
// the two roles of one kernel (fused_kernel, below):
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
// padding rows have zero queries and are ignored.  A workgroup stages the
// group's window queries in LDS once; each wave keeps them in registers when
// they fit (up to 4 row tiles) and otherwise reads them from LDS per MFMA.
// Each wave streams its key tiles through a ring of kRing one-tile buffers
// (4 KB each): while it works on one tile, the next kRing - 1 are in flight.
// The loads are unconditional (key index clamped into the range, extra tiles
// masked), so the compiler waits for exactly the tile being consumed.
//
// ML (multi-layer): grid z runs over (layer, sequence) pairs, layer-major, and
// the layer's operands come from the table; otherwise from the arguments.
#pragma once

#include "score_common.h"

namespace ckv {

// What a scoring workgroup knows before it specialises on its row-tile count.
struct Work {
  LayerView lv;
  gptr<const char> kbase;
  int layer, b, g, s0, L, P, c0, n_chunks, rt_n;
};

// Launch order of both scoring grids (one dimension).  The first part holds,
// for every (layer, sequence) and group, `lead` workgroups of cpw consecutive
// chunks; the second part holds the chunks after lead * cpw, one per
// workgroup.  The long workgroups start first and the last ones to start are
// short, so the grid drains with little idle time at its end.  In both parts
// the groups are fastest, then the key range, then the (layer, sequence) pair.
// Consecutive workgroups go to the 8 XCDs in turn, so with 8 groups a plain
// group index would give each XCD one group of every layer, and the XCDs
// would get unequal work (the number of SRHs differs between groups).  The
// group is therefore rotated by the key-range index: each XCD gets a mix of
// the groups.
struct BlockRange {
  int g, z, first, count;   // group, (layer, sequence) pair, first chunk, chunks
};

__device__ __forceinline__ BlockRange block_range(const ScoreArgs &a, int lead, int cpw,
                                                  int max_chunks) {
  const int beta = blockIdx.x;
  const int n_lead = a.Hkv * lead * a.nz;
  const bool in_lead = beta < n_lead;
  const int t = in_lead ? beta : beta - n_lead;
  const int per_z = in_lead ? lead : max_chunks - lead * cpw;   // >= 1 where reached
  const int u = t / a.Hkv;
  const int g = (t - u * a.Hkv + u) % a.Hkv;
  const int y = u % per_z, z = u / per_z;
  return in_lead ? BlockRange{g, z, y * cpw, cpw} : BlockRange{g, z, lead * cpw + y, 1};
}

// Workgroups of a scoring grid.
__host__ __device__ inline int64_t grid_blocks(int Hkv, int nz, int lead, int cpw,
                                               int max_chunks) {
  return (int64_t)Hkv * nz * (lead + (max_chunks - lead * cpw));
}

// ---------------------------------------------------------------------------
// S1+S2 partial statistics.  A workgroup (64 * kStatsWaves threads) covers
// consecutive chunks of one (sequence, group), as block_range assigns them,
// and writes one partial per chunk.  The groups of one key range are
// neighbours in launch order, so the workgroups in flight read whole token
// rows of K ([T, Hkv, D]) rather than 1/Hkv of each.
// MFMA operands: A = 16 keys, B = 16 window rows, so lane (quad, c) holds the
// logits of row c against keys 4*quad .. 4*quad+3 of the tile and keeps one
// running (ref, sum) pair per row tile.  Wave w handles the key tiles
// w, w + NW, w + 2 NW, ... of the workgroup's range; a chunk (chunk1 keys) is
// a whole number of ring turns of every wave, so its partial is the same
// whichever workgroup size covers it.
// ---------------------------------------------------------------------------
constexpr int kStatsWaves = 4;
constexpr int kStatsPartRows = 16 * 16;   // rows of the largest row-tile count (16 tiles)

// Kernels compiled for 8 or more row tiles read the query fragments one slice
// at a time (see tile_logits_all): without it they need about 296 VGPRs and
// run one wave per SIMD.  Where a row is 4 or more slices per lane, the
// statistics kernel is also held to three waves per SIMD (a few spilled
// registers); kernels for fewer row tiles are faster without either.
template <int RTM>
constexpr bool kSliceBarrier = RTM >= 8;
template <typename T, int D, int RTM>
constexpr int kStatsMinWaves = RTM >= 8 && Slices<T, D>::n >= 4 ? 3 : 1;

template <typename T, int D, int RT, bool SB, bool MARK = false>
__device__ __forceinline__ void stats_body(const ScoreArgs &a, const Work &w, uint4 *q_lds,
                                           float2 (*part)[kStatsPartRows]) {
  constexpr int NW = kStatsWaves;
  constexpr int NS = Slices<T, D>::n, RQ = RegTiles<T, D, RT>::v;
  constexpr int NT = 64 * NW;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int c = lane & 15, quad = lane >> 4;
  const int tid = threadIdx.x;
  const int c0 = w.c0, L = w.L, P = w.P, s0 = w.s0, g = w.g;
  const int tpc = a.chunk1 / (16 * NW);   // key tiles per wave and chunk (a multiple of kRing)
  const int n_tiles = tpc * w.n_chunks;
  // key row of this lane for tile index i of this wave, clamped into the range
  // (the ring's reads past the last tile hit the same cached row)
  const int k_last = min(L, c0 + w.n_chunks * a.chunk1) - 1;
  auto key_of = [&](int i) { return min(c0 + 16 * (wave + NW * i) + c, k_last); };
  float2 *parts = a.stats + w.layer * a.stats_layer +
                  ((int64_t)w.b * a.Hkv + g) * a.parts_stride * a.row_slots;

  // Query loads first, then the first kRing key tiles; the queries are written
  // to LDS while the keys are still in flight.
  uint4 qv[QStage<T, D, RT, NT>::n];
  q_load<T, D, RT, NT>(a, w.lv, w.b, w.rt_n, qv);
  uint4 kr[kRing][NS];
#pragma unroll
  for (int r = 0; r < kRing; ++r) load_k_row<T, D>(a, w.kbase, s0, key_of(r), g, quad, kr[r]);
  q_store<T, D, RT, NT>(qv, q_lds);
  __syncthreads();
  uint4 qreg[RegTiles<T, D, RT>::n][NS];
#pragma unroll
  for (int rt = 0; rt < RQ; ++rt)
#pragma unroll
    for (int s = 0; s < NS; ++s) qreg[rt][s] = q_frag<T, D>(q_lds, rt, s, c, quad);

  float ref[RT], sum[RT];
  bool ready = false;   // every row's reference is set (wave-uniform)
#pragma unroll
  for (int rt = 0; rt < RT; ++rt) {
    ref[rt] = -INFINITY;
    sum[rt] = 0.f;
  }
  auto consume = [&](const uint4 (&kf)[NS], int i) {
    f32x4 acc[RT];
    tile_logits_all<T, D, RT, true, true, SB>(kf, qreg, q_lds, c, quad, acc);
    stats_update<RT>(a, acc, ref, sum, ready, c0 + 16 * (wave + NW * i), L, P, c, quad);
  };
  // The chunk's partial: merge the four quads (same row c, different keys),
  // then the waves in order, and start the next chunk from empty pairs.
  auto flush = [&](int chunk) {
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
#pragma unroll
      for (int o = 16; o <= 32; o <<= 1) {
        float ro = __shfl_xor(ref[rt], o);
        float so = __shfl_xor(sum[rt], o);
        merge_stats(ref[rt], sum[rt], ro, so);
      }
    }
    if (quad == 0) {
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) part[wave][rt * 16 + c] = make_float2(ref[rt], sum[rt]);
    }
    __syncthreads();
    if (tid < w.rt_n * 16) {
      float r0 = part[0][tid].x, s_0 = part[0][tid].y;
#pragma unroll
      for (int v = 1; v < NW; ++v) merge_stats(r0, s_0, part[v][tid].x, part[v][tid].y);
      if constexpr (MARK) {   // published to the other workgroups of the launch
        store_partial_coherent(parts + (int64_t)chunk * a.row_slots + tid, make_float2(r0, -s_0));
      } else {
        parts[(int64_t)chunk * a.row_slots + tid] = make_float2(r0, s_0);
      }
    }
    __syncthreads();   // part is reused by the next chunk
    ready = false;
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      ref[rt] = -INFINITY;
      sum[rt] = 0.f;
    }
  };
  int chunk = c0 / a.chunk1;
  for (int i = 0; i < n_tiles; i += kRing) {
#pragma unroll
    for (int r = 0; r < kRing; ++r) {
      consume(kr[r], i + r);
      load_k_row<T, D>(a, w.kbase, s0, key_of(i + r + kRing), g, quad, kr[r]);
    }
    if ((i + kRing) % tpc == 0) flush(chunk++);   // loads of the next chunk are in flight
  }
}

template <typename T, int D, int RTM, bool ML>
__global__ __launch_bounds__(64 * kStatsWaves)
__attribute__((amdgpu_waves_per_eu(kStatsMinWaves<T, D, RTM>))) void stats_kernel(const ScoreArgs a) {
  const BlockRange r = block_range(a, a.lead1, a.cpw1, a.max_chunks1);
  Work w;
  w.g = r.g;
  w.layer = ML ? r.z / a.batch : 0;
  w.b = r.z - w.layer * a.batch;
  w.lv = layer_view<ML>(a, w.layer, w.g);
  w.kbase = w.lv.k;
  w.s0 = a.cu[w.b];
  w.L = a.cu[w.b + 1] - w.s0;
  const int chunk0 = r.first;
  if (chunk0 == 0) {   // the column-sum kernel accumulates this histogram afterwards
    int *h = a.hist + w.layer * a.hist_layer + ((int64_t)w.b * a.Hkv + w.g) * kHistBins;
    for (int i = threadIdx.x; i < kHistBins; i += 64 * kStatsWaves) h[i] = 0;
  }
  w.c0 = chunk0 * a.chunk1;
  // uniform for the whole workgroup (a group without an SRH is not scored:
  // the layer-shared index set ignores it)
  if (w.c0 >= w.L || w.lv.nsrh == 0) return;
  w.n_chunks = min(r.count, (w.L - w.c0 + a.chunk1 - 1) / a.chunk1);
  w.P = w.L - a.W;
  w.rt_n = w.lv.nsrh * a.th;

  __shared__ uint4 q_lds[RTM * 16 * QLayout<T, D>::STRIDE];
  static_assert(RTM * 16 <= kStatsPartRows, "per-wave partials of every row");
  __shared__ float2 part[kStatsWaves][kStatsPartRows];
  dispatch_rt<RTM>(w.rt_n, [&]<int RT>() { stats_body<T, D, RT, kSliceBarrier<RTM>>(a, w, q_lds, part); });
}

// ---------------------------------------------------------------------------
// S2+S3+S4.  256 threads; a workgroup covers consecutive chunks of chunk2
// keys of one (sequence, group), as block_range assigns them.
// MFMA operands: A = 16 window rows, B = 16 keys, so lane (quad, c) holds
// rows 4*quad .. 4*quad+3 of the tile against key c.  The tiles of a chunk
// plus one halo tile on each side, e = -1 .. chunk2/16, go to the waves
// round-robin (chunk2 + 32 keys = 16 * kWaves * tiles per wave and chunk);
// the ring runs on across chunks, each chunk ending with its pooling.
// ---------------------------------------------------------------------------
// Key tiles per wave in the column sums' load ring (tiles per wave and chunk,
// 16, is a multiple of it).  With the logits issued one tile ahead, two slots
// keep two tiles in flight per wave and the kernel within 256 VGPRs (two
// waves per SIMD); four slots measured slower (268 VGPRs, one wave).
constexpr int kRingCs = 2;

// FUSED: the row normalisers come from the same launch: published by the
// group's last statistics workgroup at bias_g (or, with bias_g null, merged
// here from the marked partials), polled at most `spin` more times; returns
// false, with nothing written, if they have not arrived.
template <typename T, int D, int RT, int CSW, bool SB, bool FUSED = false>
__device__ __forceinline__ bool colsum_body(const ScoreArgs &a, const Work &w, uint4 *q_lds,
                                            float *bias_s, float (*cs)[CSW], float *stage,
                                            int *hist_s, int spin = 0,
                                            const float2 *bias_g = nullptr) {
  constexpr int NS = Slices<T, D>::n, RQ = RegTiles<T, D, RT>::v;
  constexpr int NT = 64 * kWaves;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int c = lane & 15, quad = lane >> 4;
  const int tid = threadIdx.x;
  const int c0 = w.c0, L = w.L, P = w.P, s0 = w.s0, g = w.g;
  const gptr<float> out = w.lv.scores + (int64_t)g * a.T + s0;
  const int tpc = (a.chunk2 + 32) / (16 * kWaves);   // key tiles per wave and chunk
  const int n_tiles = tpc * w.n_chunks;
  // chunk, tile index e in the chunk and key row of this lane for the i-th
  // tile of this wave (clamped into the chunk and its halo)
  auto key_of = [&](int i) {
    const int ch = i / tpc;
    const int e = -1 + wave + kWaves * (i - ch * tpc);
    const int cc0 = c0 + ch * a.chunk2;
    const int k_first = max(cc0 - 16, 0), k_last = min(cc0 + a.chunk2 + 16, L) - 1;
    return min(max(cc0 + 16 * e + c, k_first), k_last);
  };

  uint4 qv[QStage<T, D, RT, NT>::n];
  q_load<T, D, RT, NT>(a, w.lv, w.b, w.rt_n, qv);
  uint4 kr[kRingCs][NS];
#pragma unroll
  for (int r = 0; r < kRingCs; ++r) load_k_row<T, D>(a, w.kbase, s0, key_of(r), g, quad, kr[r]);
  q_store<T, D, RT, NT>(qv, q_lds);
  for (int i = tid; i < kHistBins; i += NT) hist_s[i] = 0;

  // Row normalisers bias = ref + log2(sum), merged over every chunk of the
  // statistics pass; rows past the group's own get +inf.
  const float2 *parts =
      a.stats + w.layer * a.stats_layer + ((int64_t)w.b * a.Hkv + g) * a.parts_stride * a.row_slots;
  const int n_parts = (L + a.chunk1 - 1) / a.chunk1;
  if constexpr (FUSED) {
    if (bias_g != nullptr ? !read_bias_marked<NT>(bias_g, RT * 16, bias_s, spin)
                          : !merge_row_bias_marked<NT>(a, parts, a.row_slots, n_parts,
                                                       w.rt_n * 16, RT * 16, bias_s, spin))
      return false;
  } else {
    merge_row_bias<NT>(a, parts, a.row_slots, n_parts, w.rt_n * 16, RT * 16, bias_s);
  }
  __syncthreads();
  uint4 qreg[RegTiles<T, D, RT>::n][NS];
#pragma unroll
  for (int rt = 0; rt < RQ; ++rt)
#pragma unroll
    for (int s = 0; s < NS; ++s) qreg[rt][s] = q_frag<T, D>(q_lds, rt, s, c, quad);
  float bias[RT][4];
#pragma unroll
  for (int rt = 0; rt < RT; ++rt)
#pragma unroll
    for (int r = 0; r < 4; ++r) bias[rt][r] = bias_s[rt * 16 + 4 * quad + r];

  // Column sums of a chunk plus one 16-key halo tile on each side:
  // cs[h][16 + x] holds the window sum of SRH h at key cc0 + x.  The logits
  // of the wave's next tile are issued before the current tile's exp2 and
  // sums, so the matrix pipeline works while the VALU does.
  auto finish_tile = [&](const f32x4 (&lg)[RT], int i) {
    const int ch = i / tpc;
    const int cc0 = c0 + ch * a.chunk2;
    const int p_end = min(cc0 + a.chunk2, P);
    const int ntiles = (p_end - cc0 + 15) >> 4;                       // tiles e = 0 .. ntiles-1
    const int e_lo = (cc0 > 0) ? -1 : 0;                              // left halo tile
    const int e_hi = (cc0 + 16 * ntiles < P) ? ntiles : ntiles - 1;   // right halo tile
    const int e = -1 + wave + kWaves * (i - ch * tpc);
    window_sums_from_logits<RT, CSW>(a, lg, bias, e, e >= e_lo && e <= e_hi, c, quad, cs);
  };
  // Pooling of a finished chunk (S4); cs and stage are rewritten by the next
  // chunk only after every thread has pooled and stored.
  auto pool = [&](int ch) {
    const int cc0 = c0 + ch * a.chunk2;
    __syncthreads();
    pool_chunk<NT, CSW>(a, cs, w.lv.nsrh, cc0, min(cc0 + a.chunk2, P), P, out, stage, hist_s);
    __syncthreads();
  };
  // slot r of the ring holds the tiles i with i % kRingCs == r
  f32x4 lg[RT];
  tile_logits_all<T, D, RT, false, true, SB>(kr[0], qreg, q_lds, c, quad, lg);
  load_k_row<T, D>(a, w.kbase, s0, key_of(kRingCs), g, quad, kr[0]);
  for (int i = 0; i < n_tiles; i += kRingCs) {
#pragma unroll
    for (int r = 0; r < kRingCs; ++r) {
      const int rn = (r + 1) % kRingCs;   // slot of tile i + r + 1
      f32x4 lg_next[RT];
      tile_logits_all<T, D, RT, false, true, SB>(kr[rn], qreg, q_lds, c, quad, lg_next);
      load_k_row<T, D>(a, w.kbase, s0, key_of(i + r + 1 + kRingCs), g, quad, kr[rn]);
      finish_tile(lg, i + r);
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) lg[rt] = lg_next[rt];
    }
    if ((i + kRingCs) % tpc == 0) pool(i / tpc);   // loads of the next chunk are in flight
  }
  flush_hist<NT>(hist_s,
                 a.hist + w.layer * a.hist_layer + ((int64_t)w.b * a.Hkv + g) * kHistBins);
  return true;
}

template <typename T, int D, int RTM, bool ML>
__global__ __launch_bounds__(64 * kWaves) void colsum_kernel(const ScoreArgs a) {
  constexpr int NT = 64 * kWaves;
  constexpr int CSW = kMaxChunk2 + 32;
  const BlockRange r = block_range(a, a.lead2, a.cpw2, a.max_chunks2);
  Work w;
  w.g = r.g;
  w.layer = ML ? r.z / a.batch : 0;
  w.b = r.z - w.layer * a.batch;
  w.lv = layer_view<ML>(a, w.layer, w.g);
  w.kbase = w.lv.k;
  w.s0 = a.cu[w.b];
  w.L = a.cu[w.b + 1] - w.s0;
  w.c0 = r.first * a.chunk2;
  if (w.c0 >= w.L || w.lv.nsrh == 0) return;
  w.P = w.L - a.W;
  const int c_end = min(w.L, w.c0 + r.count * a.chunk2);
  // Window positions of this range are always kept: +inf.
  const gptr<float> out = w.lv.scores + (int64_t)w.g * a.T + w.s0;
  for (int j = max(w.c0, w.P) + (int)threadIdx.x; j < c_end; j += NT) out[j] = INFINITY;
  if (w.c0 >= w.P) return;                   // no prefix key in this range
  // chunks of the range that hold prefix keys
  w.n_chunks = min(r.count, (w.P - w.c0 + a.chunk2 - 1) / a.chunk2);
  w.rt_n = w.lv.nsrh * a.th;

  // The staging buffer of the pooled scores is left out where it would not fit
  // (fp32 queries with 12 row tiles); those scores are stored directly.
  constexpr size_t kLds = sizeof(uint4) * RTM * 16 * QLayout<T, D>::STRIDE +
                          sizeof(float) * (RTM * 16 + RTM * CSW + kHistBins);
  constexpr int kStage = kLds + sizeof(float) * kMaxChunk2 <= 160 * 1024 ? kMaxChunk2 : 0;
  __shared__ uint4 q_lds[RTM * 16 * QLayout<T, D>::STRIDE];
  __shared__ float bias_s[RTM * 16];
  __shared__ float cs[RTM][CSW];   // th >= 1: at most RTM SRHs
  __shared__ float stage[kStage > 0 ? kStage : 1];   // one chunk's pooled scores
  __shared__ int hist_s[kHistBins];
  dispatch_rt<RTM>(w.rt_n, [&]<int RT>() {
    colsum_body<T, D, RT, CSW, kSliceBarrier<RTM>>(a, w, q_lds, bias_s, cs,
                                                  kStage > 0 ? stage : nullptr, hist_s);
  });
}

// ---------------------------------------------------------------------------
// Both passes in one launch (fused_kernel).  Each (sequence, group) pair of
// the launch (a "segment") gets kFusedMembers statistics workgroups and as
// many column-sum workgroups.  Statistics member m computes the partials of
// a run of consecutive chunk1 chunks and publishes each with one agent-scope
// store whose sign bit is the arrival mark, then counts itself in the
// segment's arrival counter; the last to arrive merges the partials in
// merge_row_bias's order and publishes the row normalisers (marked the same
// way).  Column-sum member m waits for those and computes the column sums,
// pooling and histogram of a run of chunk2 = kFusedChunk2 chunks exactly as
// colsum_kernel does, so the normalisers, and the scores, are bit for bit
// those of the two-launch form.
// The grid interleaves the roles per XCD (fused_role): a segment's column
// sums start one block of statistics after its own, and while they run the
// next segment's statistics stream on the same CUs, so the launch has no
// drain between the passes.  A segment's workgroups are consecutive
// workgroups of one XCD (launch order goes round the 8 XCDs); that matters
// for speed only.  A column-sum workgroup whose normalisers have not arrived
// after `fused_spin` polls records itself and returns without writing:
// fused_catchup_kernel (next on the stream, when every partial is written)
// merges the partials itself and does its column sums with the same code.
// Key runs are kFusedChunk2 = 1120 (+ 32 halo keys = 9 x 128) so that 32
// members cover a 32768-key sequence's column sums.
// ---------------------------------------------------------------------------
constexpr int kFusedChunk2 = 1120;
constexpr int kFusedCsw = kFusedChunk2 + 32;

// LDS of the fused kernel; it runs where two workgroups fit a CU.  A
// workgroup has one role, so the statistics' per-wave partials share their
// space with the column sums.  The pooled-score staging buffer (STAGE) is
// left out where it would not fit (8 row tiles): those scores are stored
// directly, as colsum_kernel does in that case.
template <typename T, int D, int RTM, bool STAGE>
struct FusedLdsT {
  uint4 q[RTM * 16 * QLayout<T, D>::STRIDE];
  union {
    float2 part[kStatsWaves][kStatsPartRows];
    struct {
      float bias[RTM * 16];
      float cs[RTM][kFusedCsw];
      int hist[kHistBins];
      alignas(16) float stage[STAGE ? kFusedChunk2 + 4 : 1];
    } c;
  };
};
template <typename T, int D, int RTM>
constexpr bool kFusedStage = sizeof(FusedLdsT<T, D, RTM, true>) <= 80 * 1024;
template <typename T, int D, int RTM>
using FusedLds = FusedLdsT<T, D, RTM, kFusedStage<T, D, RTM>>;
template <typename T, int D, int RTM>
constexpr bool kFusedFits = RTM <= 8 && sizeof(FusedLds<T, D, RTM>) <= 80 * 1024;

// Segment u of the launch: the group is rotated by the (layer, sequence)
// index as in block_range.
__device__ __forceinline__ int fused_group(const ScoreArgs &a, int u) {
  const int z = u / a.Hkv;
  return (u % a.Hkv + z) % a.Hkv;
}

template <bool ML>
__device__ __forceinline__ bool fused_work(const ScoreArgs &a, int u, Work &w) {
  const int z = u / a.Hkv;
  w.g = fused_group(a, u);
  w.layer = ML ? z / a.batch : 0;
  w.b = z - w.layer * a.batch;
  w.lv = layer_view<ML>(a, w.layer, w.g);
  w.kbase = w.lv.k;
  w.s0 = a.cu[w.b];
  w.L = a.cu[w.b + 1] - w.s0;
  w.P = w.L - a.W;
  w.rt_n = w.lv.nsrh * a.th;
  return w.lv.nsrh > 0 && w.L > 0;
}

// Role of workgroup bid of the fused grid.  Each XCD (bid % 8) serves the
// segments x, x + 8, x + 16, ... (s_0 .. s_{n-1}) in blocks of kFusedMembers
// consecutive workgroups: the statistics of s_0 .. s_S, then the column sums
// of s_0 and the statistics of s_{S+1}, the column sums of s_1 and the
// statistics of s_{S+2}, ..., and finally the remaining column sums.  A
// segment's column sums thus start S blocks of statistics after its own.
constexpr int kFusedSlack = 1;
struct FusedRole {
  int u;        // segment (>= the launch's segments: nothing to do)
  int member;
  bool colsum;  // false: statistics
};
__device__ __forceinline__ FusedRole fused_role(int bid, int n_seg) {
  const int x = bid % 8, q = bid / 8;
  const int k = q / kFusedMembers;
  const int n = (n_seg - x + 7) / 8;   // segments of this XCD
  FusedRole r;
  r.member = q % kFusedMembers;
  const int A = min(kFusedSlack + 1, n);   // statistics blocks before the first column sums
  const int P = max(0, n - A);             // (column sums, statistics) pairs after them
  const int t = k - A;
  int i;
  if (k < A) {
    i = k;
    r.colsum = false;
  } else if (t < 2 * P) {
    r.colsum = (t & 1) == 0;
    i = r.colsum ? t / 2 : A + t / 2;
  } else {
    i = P + (t - 2 * P);
    r.colsum = true;
  }
  r.u = (k < 2 * n) ? x + 8 * i : n_seg;
  return r;
}

// Zeroes the partial slots the launch uses (arrival marks: the first
// max_chunks1 of each group's slots), its histograms and the catch-up list
// before the fused kernel.
static __global__ __launch_bounds__(256) void fused_fill_kernel(int *stats, int64_t n_groups,
                                                                int64_t group_stride,
                                                                int64_t group_ints, int *hist,
                                                                int64_t hist_ints, int *bias,
                                                                int64_t bias_ints, int *arrive,
                                                                int *skip) {
  const int64_t n0 = n_groups * group_ints, n1 = n0 + hist_ints, n2 = n1 + bias_ints;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n2 + n_groups;
       i += (int64_t)gridDim.x * 256) {
    if (i < n0) {
      const int64_t g = i / group_ints;
      stats[g * group_stride + (i - g * group_ints)] = 0;
    } else if (i < n1) {
      hist[i - n0] = 0;
    } else if (i < n2) {
      bias[i - n1] = 0;
    } else {
      arrive[i - n2] = 0;
    }
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) skip[0] = 0;
}

// Member `member`'s statistics chunks of segment w: published partials.
template <typename T, int D, int RTM>
__device__ __forceinline__ void fused_stats(const ScoreArgs &a, const Work &w, int u, int member,
                                            FusedLds<T, D, RTM> &sm) {
  const int n1 = (w.L + a.chunk1 - 1) / a.chunk1;
  const int c1n = (n1 + kFusedMembers - 1) / kFusedMembers;
  const int j1 = member * c1n;
  if (j1 >= n1) return;
  Work ws = w;
  ws.c0 = j1 * a.chunk1;
  ws.n_chunks = min(c1n, n1 - j1);
  dispatch_rt<RTM>(w.rt_n, [&]<int RT>() {
    stats_body<T, D, RT, kSliceBarrier<RTM>, true>(a, ws, sm.q, sm.part);
    // every partial store of this workgroup is issued (stats_body ends with a
    // barrier); the last of the segment's statistics workgroups to arrive
    // merges all partials (reading each mark) and publishes the normalisers
    __shared__ int last_s;
    if (threadIdx.x == 0)
      last_s = __hip_atomic_fetch_add(&a.fused_arrive[u], 1, __ATOMIC_RELAXED,
                                      __HIP_MEMORY_SCOPE_AGENT) ==
               (n1 + c1n - 1) / c1n - 1;
    __syncthreads();
    if (last_s) {
      const float2 *parts = a.stats + w.layer * a.stats_layer +
                            ((int64_t)w.b * a.Hkv + w.g) * a.parts_stride * a.row_slots;
      if (merge_row_bias_marked<256>(a, parts, a.row_slots, n1, w.rt_n * 16, RT * 16, sm.c.bias,
                                     1 << 16)) {
        __syncthreads();
        for (int r = threadIdx.x; r < RT * 16; r += 256)
          store_partial_coherent(a.fused_bias + (int64_t)u * a.row_slots + r,
                                 make_float2(sm.c.bias[r], -1.f));
      }
    }
  });
  __syncthreads();   // sm is reused by the next phase
}

// Member `member`'s column-sum chunks of segment w; false if a partial had
// not arrived after `spin` more polls (nothing written then).
template <typename T, int D, int RTM>
__device__ __forceinline__ bool fused_colsum(const ScoreArgs &a, const Work &w, int member,
                                             FusedLds<T, D, RTM> &sm, int spin,
                                             const float2 *bias_g) {
  const int n2 = w.P > 0 ? (w.P + a.chunk2 - 1) / a.chunk2 : 0;
  const int c2n = (n2 + kFusedMembers - 1) / kFusedMembers;
  const int j2 = member * c2n;
  if (j2 >= n2) return true;
  Work wc = w;
  wc.c0 = j2 * a.chunk2;
  wc.n_chunks = min(c2n, n2 - j2);
  bool ok = true;
  dispatch_rt<RTM>(w.rt_n, [&]<int RT>() {
    ok = colsum_body<T, D, RT, kFusedCsw, kSliceBarrier<RTM>, true>(
        a, wc, sm.q, sm.c.bias, sm.c.cs, kFusedStage<T, D, RTM> ? sm.c.stage : nullptr, sm.c.hist,
        spin, bias_g);
  });
  __syncthreads();
  return ok;
}

template <typename T, int D, int RTM, bool ML>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(2))) void fused_kernel(
    const ScoreArgs a) {
  static_assert(64 * kStatsWaves == 256 && 64 * kWaves == 256, "one workgroup shape");
  const FusedRole r = fused_role(blockIdx.x, a.nz * a.Hkv);
  if (r.u >= a.nz * a.Hkv) return;
  __shared__ FusedLds<T, D, RTM> sm;
  Work w;
  if (!fused_work<ML>(a, r.u, w)) return;
  if (!r.colsum) {
    if (r.member == 0) {   // window positions are always kept
      const gptr<float> out = w.lv.scores + (int64_t)w.g * a.T + w.s0;
      for (int j = max(w.P, 0) + (int)threadIdx.x; j < w.L; j += 256) out[j] = INFINITY;
    }
    fused_stats<T, D, RTM>(a, w, r.u, r.member, sm);
    return;
  }
  const bool done =
      a.fused_spin >= 0 && fused_colsum<T, D, RTM>(a, w, r.member, sm, a.fused_spin,
                                                   a.fused_bias + (int64_t)r.u * a.row_slots);
  if (!done && threadIdx.x == 0)
    a.fused_skip[1 + atomicAdd(&a.fused_skip[0], 1)] = r.u * kFusedMembers + r.member;
}

// The column sums the fused kernel left (entries u * kFusedMembers + member),
// after it: every partial is written by then.
template <typename T, int D, int RTM, bool ML>
__global__ __launch_bounds__(256) void fused_catchup_kernel(const ScoreArgs a) {
  __shared__ FusedLds<T, D, RTM> sm;
  const int n = a.fused_skip[0];
  for (int i = blockIdx.x; i < n; i += gridDim.x) {
    const int e = a.fused_skip[1 + i];
    Work w;
    fused_work<ML>(a, e / kFusedMembers, w);
    fused_colsum<T, D, RTM>(a, w, e % kFusedMembers, sm, 0, nullptr);
  }
}

// ---------------------------------------------------------------------------
// Host-side launcher template; grid z = batch * n_layers (n_layers = 1 unless ML).
// ---------------------------------------------------------------------------
template <typename T, int D, int RTM, bool ML>
static hipError_t launch_score_t(const ScoreArgs &args, int nz, hipStream_t stream) {
  ScoreArgs a = args;
  a.nz = nz;
  if (a.fused_skip != nullptr) {
    if constexpr (kFusedFits<T, D, RTM>) {
      a.chunk2 = kFusedChunk2;   // the column-sum runs of the fused grid
      const int n_layers = ML ? nz / a.batch : 1;
      const int64_t nb = fused_blocks(a.Hkv, nz);
      if (nb > INT32_MAX) return hipErrorInvalidConfiguration;
      const int64_t slots = (int64_t)a.parts_stride * a.row_slots * 2;   // ints per group
      const int64_t n_groups = (int64_t)n_layers * a.batch * a.Hkv;
      hipLaunchKernelGGL(fused_fill_kernel, dim3(1024), dim3(256), 0, stream,
                         reinterpret_cast<int *>(a.stats), n_groups, slots,
                         (int64_t)a.max_chunks1 * a.row_slots * 2, a.hist,
                         (int64_t)a.hist_layer * n_layers, reinterpret_cast<int *>(a.fused_bias),
                         n_groups * a.row_slots * 2, a.fused_arrive, a.fused_skip);
      hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
      hipLaunchKernelGGL((fused_kernel<T, D, RTM, ML>), dim3((unsigned)nb), dim3(256), 0, stream,
                         a);
      if ((e = hipGetLastError()) != hipSuccess) return e;
      hipLaunchKernelGGL((fused_catchup_kernel<T, D, RTM, ML>), dim3(64), dim3(256), 0, stream, a);
      return hipGetLastError();
    } else {
      return hipErrorInvalidConfiguration;   // the host plans the fused launch only where it fits
    }
  }
  const int64_t n1 = grid_blocks(a.Hkv, nz, a.lead1, a.cpw1, a.max_chunks1);
  const int64_t n2 = grid_blocks(a.Hkv, nz, a.lead2, a.cpw2, a.max_chunks2);
  if (n1 < 1 || n2 < 1 || n1 > INT32_MAX || n2 > INT32_MAX) return hipErrorInvalidConfiguration;
  hipLaunchKernelGGL((stats_kernel<T, D, RTM, ML>), dim3((unsigned)n1), dim3(64 * kStatsWaves),
                     0, stream, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((colsum_kernel<T, D, RTM, ML>), dim3((unsigned)n2), dim3(64 * kWaves), 0,
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
    case 9:
    case 10:
    case 11:
    case 12: return launch_score_t<T, D, 12, ML>(a, nz, stream);
    default:
      // 16 row tiles of fp32 queries at D = 128 do not fit the LDS (the host
      // caps that shape at 12)
      if constexpr (sizeof(T) * D <= 256) return launch_score_t<T, D, 16, ML>(a, nz, stream);
      return hipErrorInvalidConfiguration;
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
