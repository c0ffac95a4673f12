// Single-pass scoring (steps S1-S4) for gfx950: every key is read from HBM once.
//
// The window softmax (section 3.3, with the SnapKV observation window of
// section 4) needs each window row's normaliser over the whole sequence
// before any column sum can be formed.  Here a unit of 256 keys of one
// (layer, sequence, KV group) -- a "segment" -- is scored in two steps that
// run at different times in the same workgroup:
//
//   statistics  the logits of every SRH window row against the unit's keys
//               (bf16 MFMA, A = keys, B = window rows: a lane holds one row
//               and four keys of each tile) are turned into e = exp2(y - ref)
//               with a per-lane, per-row reference ref, and kept in
//               registers; the unit's partial (max, sum) per row is published
//               to the workspace;
//   finish      once every unit of the segment has published, the last one
//               to arrive merges the partials into each row's normaliser
//               bias = ref_row + log2(sum_row) and publishes it; the
//               unit's window sums are then sum_rows e * exp2(ref - bias)
//               (one multiply-add per logit, no second MFMA or exp), pooled
//               along the token axis in LDS and averaged over the SRHs.
//
// Persistent workgroups of 8 waves (one per CU) take units from an atomic
// ticket, numbered layer by layer, sequence by sequence and group by group,
// so a segment's units are taken close together in time.  A workgroup runs
// a three-stage pipeline: in the iteration that computes unit k's statistics
// it finishes unit k-2 and has the keys of units k+1 and k+2 in flight, so a
// segment's normaliser has two iterations to arrive.  The wait for it is
// bounded; a unit whose normaliser has not arrived is appended to a list and
// finished by onepass_catchup_kernel, which runs next on the same stream and
// recomputes exactly the same values (same device code, same order of every
// sum), so results never depend on timing.
//
// Pooling needs window sums on both sides of a position.  A unit pools the
// positions whose pooling window lies inside it; the 2r positions around each
// boundary between two units are pooled by onepass_boundary_kernel from the
// window sums both units store at their ends.
//
// Published values carry a marker: a unit partial is stored as (max, -sum)
// (the sign bit is the marker; the workspace is zeroed first), a normaliser
// as (bias, 1).  The merger waits (bounded) for partials whose stores are
// still in flight, so no unit ever waits for its own stores to complete.
#include "ckv_launch.h"
#include "score_common.h"

namespace ckv {

constexpr int kOpWaves = 8;
constexpr int kOpThreads = 64 * kOpWaves;
constexpr int kOpTiles = 2;                          // key tiles per wave and unit
constexpr int kOpUnit = 16 * kOpWaves * kOpTiles;    // keys per unit
constexpr int kOpMergeBatch = 8;                     // partial loads in flight per merging thread

static_assert(kOpUnit == kOnePassUnitKeys, "unit size shared with the host plan");

__global__ __launch_bounds__(256) void op_fill_kernel(int *p, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (int64_t)gridDim.x * 256)
    p[i] = 0;
}

// A unit, decoded from its ticket (workgroup-uniform).
struct OpUnit {
  int valid;
  int ticket, layer, b, g, u, n_u, s0, L, P, u0, gi, seg, nh, rt_n;
  int first_ticket;   // ticket of unit 0 of the segment
};

// UNIFORM: the ticket is the same in every lane (the decode then stays in
// scalar registers); the boundary kernel decodes a different unit per lane.
template <bool UNIFORM = true>
__device__ __forceinline__ OpUnit op_decode(const OnePassArgs &f, int ticket_any) {
  const ScoreArgs &a = f.s;
  const int tk_in = UNIFORM ? __builtin_amdgcn_readfirstlane(ticket_any) : ticket_any;
  OpUnit x{};
  x.valid = tk_in >= 0 && tk_in < f.n_units_total;
  // an invalid ticket decodes as unit 0 (valid addresses for the loads that
  // every iteration issues unconditionally; nothing of it is used)
  const int tk = x.valid ? tk_in : 0;
  x.ticket = tk_in;
  x.layer = tk / f.units_per_layer;
  const int t = tk - x.layer * f.units_per_layer;
  int b = 0;
  while (b + 1 < a.batch && f.seq_units[b + 1] <= t) ++b;
  x.b = b;
  const cptr<int32_t> cu = to_const(a.cu);
  x.s0 = cu[b];
  x.L = cu[b + 1] - x.s0;
  x.n_u = (x.L + kOpUnit - 1) / kOpUnit;
  x.g = (t - f.seq_units[b]) / x.n_u;
  x.u = (t - f.seq_units[b]) - x.g * x.n_u;
  x.first_ticket = tk - x.u;
  x.P = x.L - a.W;
  x.u0 = x.u * kOpUnit;
  x.gi = b * a.Hkv + x.g;
  x.seg = x.layer * a.batch * a.Hkv + x.gi;
  x.nh = srh_count<true>(a, x.layer, x.g);
  x.rt_n = x.nh * a.th;
  return x;
}

__device__ __forceinline__ bool op_in_segment(const OpUnit &x, int ticket) {
  return ticket >= x.first_ticket && ticket < x.first_ticket + x.n_u;
}

// The unit partials of segment x: [unit][row_slots] (max, -sum).
__device__ __forceinline__ float2 *op_partials(const ScoreArgs &a, const OpUnit &x) {
  return a.stats + x.layer * a.stats_layer + (int64_t)x.gi * a.parts_stride * a.row_slots;
}

// The global loads of unit x (decoded from any ticket, valid or not): its
// window queries, then its keys (tiles wave and wave + 8 of the unit).  Every
// load is issued, with indices clamped into range, so that each wave issues
// the same number of loads on every path; the values of rows a group does not
// have, and of padding rows, are replaced by zeros.  The compiler can then
// count exactly how many loads follow an earlier one, and a wait for an
// earlier value never waits for these.
template <typename T, int D, int RTM>
__device__ __forceinline__ void op_unit_loads(const ScoreArgs &a, const OpUnit &x,
                                              uint4 (&kr)[kOpTiles][Slices<T, D>::n],
                                              uint4 (&qv)[QStage<T, D, RTM, kOpThreads>::n]) {
  constexpr int U4 = QLayout<T, D>::U4;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int c = lane & 15, quad = lane >> 4;
  const LayerView lv = layer_view<true>(a, x.layer, x.g);
  const int rt_n = max(x.rt_n, 1);
  // the group's SRH heads (at most RTM) from the table's srh_head bytes,
  // three aligned words read as scalars
  const cptr<LayerDesc> d = to_const(a.layers) + x.layer;
  const cptr<uint32_t> hw = reinterpret_cast<cptr<uint32_t>>(
      reinterpret_cast<cptr<char>>(d) + offsetof(LayerDesc, srh_head));
  const int w0 = min(lv.off >> 2, kMaxQHeads / 4 - 3);
  const uint32_t hw0 = hw[w0], hw1 = hw[w0 + 1], hw2 = hw[w0 + 2];
#pragma unroll
  for (int it = 0; it < QStage<T, D, RTM, kOpThreads>::n; ++it) {
    const int idx = (int)threadIdx.x + it * kOpThreads;
    const int row = idx / U4, u = idx - row * U4;
    const int rt = row >> 4;
    const int rtc = min(rt, rt_n - 1);
    const int i = (rtc % a.th) * 16 + (row & 15);
    const int ic = min(i, a.W - 1);
    const int byte = lv.off + rtc / a.th - 4 * w0;   // < 12 for at most 6 heads
    const uint32_t word = byte < 4 ? hw0 : byte < 8 ? hw1 : hw2;
    const int head = (int)((word >> (8 * (byte & 3))) & 0xFFu);
    const uint4 v = load16(lv.q + (((int64_t)x.b * a.W + ic) * a.Hq + head) *
                                      (int64_t)(D * sizeof(T)) + 16 * u);
    const bool real = rt < x.rt_n && i < a.W && row < RTM * 16;
    qv[it] = real ? v : make_uint4(0, 0, 0, 0);
  }
#pragma unroll
  for (int t = 0; t < kOpTiles; ++t)
    load_k_row<T, D>(a, lv.k, x.s0, max(0, min(x.u0 + 16 * (wave + kOpWaves * t) + c, x.L - 1)),
                     x.g, quad, kr[t]);
}

// Whether key j is visible to the window row of lane row c in row tile rt:
// inside the sequence and, for a window row i, at most its own position P + i.
__device__ __forceinline__ bool op_visible(const ScoreArgs &a, int rt, int c, int j, int L,
                                           int P) {
  const int i = (rt % a.th) * 16 + c;
  return (j < L) && (i >= a.W || j <= P + i);
}

// e-values of the first tile of a unit, in place (lane: row c of each row
// tile, keys base + 4*quad + r): the reference of a row is the largest of the
// lane's visible logits y (base-2 units), e = exp2(y - ref),
// sum = ((e0 + e1) + e2) + e3.  Invisible keys get e = 0; a row with no
// visible key keeps ref = -inf and sum = 0.
template <int RTM, bool MASKED>
__device__ __forceinline__ void ev_first(const ScoreArgs &a, int rtu, f32x4 (&e)[RTM],
                                         float (&ref)[RTM], float (&sum)[RTM], int base, int L,
                                         int P, int c, int quad) {
#pragma unroll
  for (int rt = 0; rt < RTM; ++rt) {
    if (rt < rtu) {
      float m = -INFINITY;
  #pragma unroll
      for (int r = 0; r < 4; ++r) {
        if (MASKED && !op_visible(a, rt, c, base + 4 * quad + r, L, P)) e[rt][r] = -INFINITY;
        else e[rt][r] *= a.c1;
        m = fmaxf(m, e[rt][r]);
      }
      ref[rt] = m;
      const float mm = (m == -INFINITY) ? 0.f : m;   // all -inf: every term exp2(-inf) = 0
  #pragma unroll
      for (int r = 0; r < 4; ++r) e[rt][r] = fast_exp2(e[rt][r] - mm);
      sum[rt] = ((e[rt][0] + e[rt][1]) + e[rt][2]) + e[rt][3];
      __builtin_amdgcn_sched_barrier(0);
    }
  }
}

// e-values of a later tile, in place, against the running reference.  A row
// whose new terms would exceed 2^30 (or that had no visible key yet) is
// rebased on its largest new logit, and the unit's earlier e-values and its
// sum are rescaled.
template <int RTM, bool MASKED>
__device__ __forceinline__ void ev_next(const ScoreArgs &a, int rtu, f32x4 (&e)[RTM],
                                        f32x4 (&e_prev)[RTM], float (&ref)[RTM],
                                        float (&sum)[RTM], int base, int L, int P, int c,
                                        int quad) {
  constexpr float kRescale = 30.f;
#pragma unroll
  for (int rt = 0; rt < RTM; ++rt) {
    if (rt < rtu) {
      // d = y - ref (= y while the row has no reference yet)
      const float nref = (ref[rt] == -INFINITY) ? 0.f : -ref[rt];
      float dm = -INFINITY;
  #pragma unroll
      for (int r = 0; r < 4; ++r) {
        if (MASKED && !op_visible(a, rt, c, base + 4 * quad + r, L, P)) e[rt][r] = -INFINITY;
        else e[rt][r] = __builtin_fmaf(e[rt][r], a.c1, nref);
        dm = fmaxf(dm, e[rt][r]);
      }
      if (dm > kRescale || (ref[rt] == -INFINITY && dm != -INFINITY)) {   // rare, per lane
        const float f = (ref[rt] == -INFINITY) ? 0.f : fast_exp2(-dm);
        sum[rt] *= f;
  #pragma unroll
        for (int r = 0; r < 4; ++r) e_prev[rt][r] *= f;
        ref[rt] = (ref[rt] == -INFINITY) ? dm : ref[rt] + dm;
  #pragma unroll
        for (int r = 0; r < 4; ++r) e[rt][r] -= dm;
      }
  #pragma unroll
      for (int r = 0; r < 4; ++r) e[rt][r] = fast_exp2(e[rt][r]);
      sum[rt] += ((e[rt][0] + e[rt][1]) + e[rt][2]) + e[rt][3];
      __builtin_amdgcn_sched_barrier(0);
    }
  }
}

// S1 of unit x: logits of both key tiles of this wave (query fragments read
// once per slice and row tile) into e.  Then S2 (op_unit_stats): their
// e-values, and the unit's partial (max, sum) per row merged over the quads
// and waves.  Threads r < rt_n * 16 return row r's partial; mu_s[r] receives
// the unit's max of row r, and the e-values are rescaled to it
// (e = exp2(y - mu)), so that a unit is finished from its e-values and mu_s
// alone.  Ends with `part` free again.
template <typename T, int D, int RTM>
__device__ __forceinline__ void op_unit_logits(const OpUnit &x,
                                               const uint4 (&kr)[kOpTiles][Slices<T, D>::n],
                                               const uint4 *q_lds, f32x4 (&e)[kOpTiles][RTM]) {
  constexpr int NS = Slices<T, D>::n;
  const int lane = threadIdx.x & 63;
  const int c = lane & 15, quad = lane >> 4;
  const int rtu = rt_class(x.rt_n);   // row tiles computed (the extra ones have zero queries)
  // one slice's query fragments in flight at a time (the compiler would
  // otherwise read all of them from LDS ahead of the MFMAs)
#pragma unroll
  for (int s = 0; s < NS; ++s) {
#pragma unroll
    for (int rt = 0; rt < RTM; ++rt) {
      if (rt < rtu) {
        const uint4 qf = q_frag<T, D>(q_lds, rt, s, c, quad);
  #pragma unroll
        for (int t = 0; t < kOpTiles; ++t)
          e[t][rt] = mfma_slice<T>(kr[t][s], qf, s == 0 ? f32x4{0.f, 0.f, 0.f, 0.f} : e[t][rt]);
      }
    }
    __builtin_amdgcn_sched_barrier(0);
  }
}

template <int RTM>
__device__ __forceinline__ float2 op_unit_stats(const ScoreArgs &a, const OpUnit &x,
                                                f32x4 (&e)[kOpTiles][RTM], float *mu_s,
                                                float2 (*part)[RTM * 16]) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int c = lane & 15, quad = lane >> 4;
  const int rtu = rt_class(x.rt_n);
  float ref[RTM], sum[RTM];
  const int base0 = x.u0 + 16 * wave;
  if (base0 + 16 <= x.P)
    ev_first<RTM, false>(a, rtu, e[0], ref, sum, base0, x.L, x.P, c, quad);
  else
    ev_first<RTM, true>(a, rtu, e[0], ref, sum, base0, x.L, x.P, c, quad);
#pragma unroll
  for (int t = 1; t < kOpTiles; ++t) {
    const int base = x.u0 + 16 * (wave + kOpWaves * t);
    if (base + 16 <= x.P)
      ev_next<RTM, false>(a, rtu, e[t], e[t - 1], ref, sum, base, x.L, x.P, c, quad);
    else
      ev_next<RTM, true>(a, rtu, e[t], e[t - 1], ref, sum, base, x.L, x.P, c, quad);
  }
  // merge the four quads (same row c, other keys), then the waves in order
#pragma unroll
  for (int rt = 0; rt < RTM; ++rt) {
    if (rt < rtu) {
      float m = ref[rt], sm = sum[rt];
  #pragma unroll
      for (int o = 16; o <= 32; o <<= 1) {
        const float mo = __shfl_xor(m, o), so = __shfl_xor(sm, o);
        merge_stats(m, sm, mo, so);
      }
      if (quad == 0) part[wave][rt * 16 + c] = make_float2(m, sm);
    }
  }
  __syncthreads();
  float2 res = make_float2(-INFINITY, 0.f);
  if (tid < rtu * 16) {
    float m = part[0][tid].x, sm = part[0][tid].y;
#pragma unroll
    for (int w = 1; w < kOpWaves; ++w) merge_stats(m, sm, part[w][tid].x, part[w][tid].y);
    res = make_float2(m, sm);
    mu_s[tid] = m;
  }
  __syncthreads();   // part is reused; mu_s is complete
  // e = exp2(y - ref) * exp2(ref - mu) (a row without visible keys: 0)
#pragma unroll
  for (int rt = 0; rt < RTM; ++rt) {
    if (rt < rtu) {
      const float mu = mu_s[rt * 16 + c];
      const float f = (ref[rt] == -INFINITY) ? 0.f : fast_exp2(ref[rt] - mu);
  #pragma unroll
      for (int t = 0; t < kOpTiles; ++t) e[t][rt] *= f;
    }
  }
  return res;
}

// Row normalisers of segment x from its n_u unit partials, merged in unit
// order per thread and then over tpr threads per row (a fixed tree), into
// bias_s; rows past the group's own (or past W inside a row tile) get +inf.
// With spin > 0 a partial whose marker is not set yet is read again, at most
// `spin` times; returns false (uniformly) if one never arrived.
__device__ __forceinline__ bool op_merge_segment(const ScoreArgs &a, const OpUnit &x, int spin,
                                                 int rows_cap, float *bias_s) {
  const int tid = threadIdx.x;
  const int rows = x.rt_n * 16;
  const float2 *parts = op_partials(a, x);
  int tpr = 1;
  while (tpr * 2 * rows <= kOpThreads && tpr < 32) tpr *= 2;
  const int row = tid / tpr, sub = tid % tpr;
  float m = -INFINITY, sm = 0.f;
  bool ok = true;
  if (row < rows) {
    for (int k0 = sub; k0 < x.n_u; k0 += kOpMergeBatch * tpr) {
      float2 v[kOpMergeBatch];
#pragma unroll
      for (int j = 0; j < kOpMergeBatch; ++j) {
        const int k = min(k0 + j * tpr, x.n_u - 1);
        v[j] = load_partial_coherent(parts + (int64_t)k * a.row_slots + row);
      }
#pragma unroll
      for (int j = 0; j < kOpMergeBatch; ++j) {
        if (k0 + j * tpr >= x.n_u) continue;
        int tries = 0;
        while (!signbit(v[j].y) && tries < spin) {
          __builtin_amdgcn_s_sleep(2);
          v[j] = load_partial_coherent(parts + (int64_t)(k0 + j * tpr) * a.row_slots + row);
          ++tries;
        }
        ok = ok && signbit(v[j].y);
        merge_stats(m, sm, v[j].x, -v[j].y);
      }
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
  for (int r = rows + tid; r < rows_cap; r += kOpThreads) bias_s[r] = INFINITY;
  return __syncthreads_and(ok);
}

template <int CTRL>
__device__ __forceinline__ float dpp_f(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, false));
}

// Sum over the 16 lanes c of one quad of v[r(c)], where lane c ends up with
// key r(c) = 2 (c & 1) + ((c >> 1) & 1): pairwise exchanges halve the values
// a lane carries (c ^ 1, then c ^ 2), then lanes c, c + 4, c + 8, c + 12 are
// added.  Lanes c < 4 hold the four keys; the order of every sum is fixed.
__device__ __forceinline__ float quad_rows_to_keys(const float (&v)[4], int c) {
  const bool o1 = (c & 1) != 0, o2 = (c & 2) != 0;
  const float k0 = o1 ? v[2] : v[0], k1 = o1 ? v[3] : v[1];
  const float s0 = o1 ? v[0] : v[2], s1 = o1 ? v[1] : v[3];
  const float a0 = k0 + dpp_f<0xB1>(s0);   // quad_perm [1, 0, 3, 2]: lane c ^ 1
  const float a1 = k1 + dpp_f<0xB1>(s1);
  const float kk = o2 ? a1 : a0, ss = o2 ? a0 : a1;
  float b = kk + dpp_f<0x4E>(ss);           // quad_perm [2, 3, 0, 1]: lane c ^ 2
  b += dpp_f<0x124>(b);                     // row_ror 4
  b += dpp_f<0x128>(b);                     // row_ror 8
  return b;
}

// Pooled, SRH-averaged score of prefix position x0 + j from window sums
// cs_at(h, x) (x = position), pooling window clipped to [0, P).
template <typename F>
__device__ __forceinline__ float op_pool(const ScoreArgs &a, F cs_at, int nh, int pos, int P) {
  const int rp = (a.pool_kernel - 1) >> 1;
  const int lo = max(pos - rp, 0), hi = min(pos + rp, P - 1);
  const float inv_k = 1.f / (float)a.pool_kernel;
  const float inv_n = 1.f / (float)nh;
  float score;
  if (a.reduce_order == 0) {          // pool each SRH, then average
    score = 0.f;
    for (int h = 0; h < nh; ++h) {
      float v;
      if (a.pool_type == 0) {
        v = -INFINITY;
        for (int x = lo; x <= hi; ++x) v = fmaxf(v, cs_at(h, x));
      } else {
        v = 0.f;
        for (int x = lo; x <= hi; ++x) v += cs_at(h, x);
        v *= inv_k;
      }
      score += v;
    }
    score *= inv_n;
  } else {                            // average the SRH sums, then pool
    score = (a.pool_type == 0) ? -INFINITY : 0.f;
    for (int x = lo; x <= hi; ++x) {
      float m = 0.f;
      for (int h = 0; h < nh; ++h) m += cs_at(h, x);
      score = (a.pool_type == 0) ? fmaxf(score, m * inv_n) : score + m * inv_n;
    }
    if (a.pool_type != 0) score *= inv_k;
  }
  return score;
}

// S3 + S4 of unit x from its e-values and row maxima mu_s, with the segment's
// normalisers in bias_s, into LDS only: window sums per SRH into cs, the
// pooled scores of the unit's interior positions into stage (and their
// first-digit histogram into hist2, two 16-bit counts per word, at most 256
// per unit), and the window sums of the unit's first and last ew keys into
// edge_s ([h][side][ew]: side 0 = keys u0 .. u0 + ew - 1, side 1 = the last ew
// keys) for the boundary kernel.  op_unit_flush writes them out.  Starts and
// ends with a barrier-separated use of cs.
template <int RTM>
__device__ __forceinline__ void op_unit_finish(const OnePassArgs &f, const OpUnit &x,
                                               const f32x4 (&e)[kOpTiles][RTM],
                                               const float *mu_s, const float *bias_s,
                                               float (*cs)[kOpUnit], float *stage, float *edge_s,
                                               uint32_t *hist2) {
  const ScoreArgs &a = f.s;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int c = lane & 15, quad = lane >> 4;
  const int rtu = rt_class(x.rt_n);
  const int rsel = 2 * (c & 1) + ((c >> 1) & 1);
#pragma unroll
  for (int t = 0; t < kOpTiles; ++t) {
    const int key0 = 16 * (wave + kOpWaves * t) + 4 * quad;
    int h = 0;
    float v[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int rt = 0; rt < RTM; ++rt) {
      if (rt < rtu) {
        const float w = fast_exp2(mu_s[rt * 16 + c] - bias_s[rt * 16 + c]);
        const bool first = rt == 0 || ((a.head_end_mask >> (rt - 1)) & 1u);
#pragma unroll
        for (int r = 0; r < 4; ++r)
          v[r] = first ? e[t][rt][r] * w : __builtin_fmaf(e[t][rt][r], w, v[r]);
        if ((a.head_end_mask >> rt) & 1u) {
          const float sv = quad_rows_to_keys(v, c);
          if (c < 4) cs[h][key0 + rsel] = sv;
          ++h;
        }
      }
    }
  }
  __syncthreads();
  const int rp = (a.pool_kernel - 1) >> 1;
  auto cs_at = [&](int h, int pos) { return cs[h][pos - x.u0]; };
  for (int j = tid; j < kOpUnit; j += kOpThreads) {
    const int pos = x.u0 + j;
    if (pos >= x.P) continue;
    const bool left_ok = x.u == 0 || pos - rp >= x.u0;
    const bool right_ok = pos + rp < x.u0 + kOpUnit || x.P <= x.u0 + kOpUnit;
    if (!(left_ok && right_ok)) continue;   // pooled by the boundary kernel
    const float score = op_pool(a, cs_at, x.nh, pos, x.P);
    stage[j] = score;
    const int bin = hist_bin(__float_as_uint(score));
    atomicAdd(&hist2[bin >> 1], 1u << (16 * (bin & 1)));
  }
  const int ew = f.ew;
  for (int i = tid; i < x.nh * 2 * ew; i += kOpThreads) {
    const int h = i / (2 * ew), side = (i / ew) & 1, k = i % ew;
    edge_s[i] = cs[h][side ? kOpUnit - ew + k : k];
  }
  __syncthreads();   // cs is reused
}

// The global writes of a unit: its scores (the interior positions op_unit_finish
// pooled, +inf on window positions; WINDOW_ONLY: a unit without prefix
// positions), its edge window sums and its histogram counts (which are
// cleared in LDS).  The positions within r of a boundary with another unit
// are written by the boundary kernel.
template <bool WINDOW_ONLY>
__device__ __forceinline__ void op_unit_flush(const OnePassArgs &f, const OpUnit &x,
                                              const float *stage, const float *edge_s,
                                              uint32_t *hist2) {
  const ScoreArgs &a = f.s;
  const int tid = threadIdx.x;
  const LayerView lv = layer_view<true>(a, x.layer, x.g);
  const gptr<float> out = lv.scores + (int64_t)x.g * a.T + x.s0;
  const int rp = (a.pool_kernel - 1) >> 1;
  const int u_end = min(x.u0 + kOpUnit, x.L);
  for (int j = tid; j < kOpUnit; j += kOpThreads) {
    const int pos = x.u0 + j;
    if (pos >= u_end) continue;
    if (WINDOW_ONLY || pos >= x.P) {
      out[pos] = INFINITY;
      continue;
    }
    const bool left_ok = x.u == 0 || pos - rp >= x.u0;
    const bool right_ok = pos + rp < x.u0 + kOpUnit || x.P <= x.u0 + kOpUnit;
    if (left_ok && right_ok) out[pos] = stage[j];
  }
  if constexpr (WINDOW_ONLY) return;
  const int ew = f.ew;
  float *ed = f.edges + (int64_t)x.ticket * f.heads_max * 2 * ew;
  for (int i = tid; i < x.nh * 2 * ew; i += kOpThreads) ed[i] = edge_s[i];
  int *hg = a.hist + x.layer * a.hist_layer + (int64_t)x.gi * kHistBins;
  for (int i = tid; i < kHistBins / 2; i += kOpThreads) {
    const uint32_t n = hist2[i];
    if (n) {
      if (n & 0xFFFFu) atomicAdd(&hg[2 * i], (int)(n & 0xFFFFu));
      if (n >> 16) atomicAdd(&hg[2 * i + 1], (int)(n >> 16));
      hist2[i] = 0;
    }
  }
}

// LDS of the single-pass kernels, kept under 64 KiB so that every access is a
// base register plus an instruction offset.  The partial statistics of the
// statistics step and the window sums of the finish step are never live at
// the same time and share their space.
template <typename T, int D, int RTM, int NQ>
struct OpLds {
  uint4 q[NQ][RTM * 16 * QLayout<T, D>::STRIDE];   // window queries of the next units
  union {
    float2 part[kOpWaves][RTM * 16];
    float cs[RTM][kOpUnit];
  } u;
  float bias_s[RTM * 16];
  float mu_s[2][RTM * 16];
  float stage[kOpUnit];                          // pooled scores of the unit being finished
  float edge_s[RTM * 2 * (kMaxPoolKernel - 1)];  // its edge window sums
  uint32_t hist2[kHistBins / 2];
  int tk_s[4];
};

// Main kernel: persistent workgroups (at most one per CU), see the header.
// Iteration k: A = unit k - 2 is finished from e-value set k % 2, then
// B = unit k's logits go into the same set; unit k - 1 waits in the other
// set.  Unit k + 1's keys and queries are loaded into the registers B's
// operands came from as soon as B's MFMAs have read them.  Every global load
// or atomic whose result is needed is issued about an iteration before its
// use (the vector-memory counter completes in order, so an early use would
// also wait for the key loads issued after it).
template <typename T, int D, int RTM>
__global__ __launch_bounds__(kOpThreads) void onepass_kernel(const OnePassArgs f) {
  constexpr int NS = Slices<T, D>::n;
  constexpr int QN = QStage<T, D, RTM, kOpThreads>::n;
  const ScoreArgs &a = f.s;
  const int tid = threadIdx.x;

  __shared__ OpLds<T, D, RTM, 1> sm;
  static_assert(sizeof(OpLds<T, D, RTM, 1>) <= 65536, "LDS offsets must fit 16 bits");
  uint4 *q_lds = sm.q[0];
  auto &part = sm.u.part;
  auto &cs = sm.u.cs;
  float *bias_s = sm.bias_s;
  auto &mu_s = sm.mu_s;
  uint32_t *hist2 = sm.hist2;
  int *tk_s = sm.tk_s;

  uint4 kr[kOpTiles][NS];              // keys of the next unit to score
  f32x4 ev[2][kOpTiles][RTM];          // e-values of units k - 1 and k (k - 2 before B)
  uint4 qv[QN];                        // its window queries
  float2 pv = make_float2(0.f, 0.f);   // polled normaliser of the next unit to finish
  int arrived = -1;                    // thread 0: arrival count before the last publication
  int tk_req = -1;                     // thread 0: ticket requested for the next unit

  for (int i = tid; i < kHistBins / 2; i += kOpThreads) hist2[i] = 0;
  if (tid == 0) {
    tk_s[0] = atomicAdd(f.ticket, 1);
    tk_req = atomicAdd(f.ticket, 1);
  }
  __syncthreads();
  int tA = -1, tA2 = -1, tB = tk_s[0];
  int t_pub = -1;   // unit published in the previous iteration (its arrival is checked next)
  op_unit_loads<T, D, RTM>(a, op_decode(f, tB), kr, qv);

  auto iterate = [&]<int P>() __attribute__((always_inline)) -> bool {
    // 1. the previous publication: if it was its segment's last arrival, merge
    //    and publish the segment's normalisers before anything that may wait
    //    (so that no workgroup's wait delays another segment's merge); the
    //    ticket of unit k + 1
    if (tid == 0) {
      tk_s[2] = (t_pub >= 0) ? arrived : -1;
      tk_s[3] = tk_req;
    }
    __syncthreads();
    const int tC = tk_s[3];
    if (t_pub >= 0) {
      const OpUnit X = op_decode(f, t_pub);
      if (tk_s[2] == X.n_u - 1) {
        if (op_merge_segment(a, X, 1 << 16, RTM * 16, bias_s)) {
          if (tid < X.rt_n * 16)
            store_partial_coherent(f.bias + (int64_t)X.seg * a.row_slots + tid,
                                   make_float2(bias_s[tid], 1.f));
        }
      }
    }
    // 2. finish A = unit k - 2 (its normalisers were polled an iteration ago)
    //    into LDS; its global writes follow B's logits (step 4), so that the
    //    wait for B's keys does not wait for them
    const OpUnit A = op_decode(f, tA);
    int flush = 0;   // 1: A finished, 2: A has only window positions
    if (A.valid) {
      if (A.u0 < A.P) {
        const int rows = A.rt_n * 16;
        // a unit this workgroup has not published yet can not arrive while it
        // waits: A is finished later if B or unit k + 1 belongs to A's segment
        const bool self = op_in_segment(A, tB) || op_in_segment(A, tC);
        int ok = __syncthreads_and((tid >= rows || pv.y == 1.f) && f.spin_limit >= 0);
        for (int spins = 0; !ok && !self && spins < f.spin_limit; ++spins) {
          __builtin_amdgcn_s_sleep(8);
          if (tid < rows)
            pv = load_partial_coherent(f.bias + (int64_t)A.seg * a.row_slots + tid);
          ok = __syncthreads_and(tid >= rows || pv.y == 1.f);
        }
        if (ok) {
          if (tid < rows) bias_s[tid] = pv.x;
          for (int r = rows + tid; r < RTM * 16; r += kOpThreads) bias_s[r] = INFINITY;
          __syncthreads();
          op_unit_finish<RTM>(f, A, ev[P], mu_s[P], bias_s, cs, sm.stage, sm.edge_s, hist2);
          flush = 1;
        } else if (tid == 0) {
          f.skip_list[atomicAdd(f.skip_count, 1)] = A.ticket;
        }
      } else {
        flush = 2;
      }
    }
    // 3. B's queries to LDS
    const OpUnit B = op_decode(f, tB);
    if (B.valid) q_store<T, D, RTM, kOpThreads>(qv, q_lds);
    __syncthreads();
    // 4. B = unit k: logits; A's global writes; the poll of unit k - 1's
    //    normalisers (finished in the next iteration)
    t_pub = -1;
    if (B.valid) op_unit_logits<T, D, RTM>(B, kr, q_lds, ev[P]);
    if (flush == 1) op_unit_flush<false>(f, A, sm.stage, sm.edge_s, hist2);
    if (flush == 2) op_unit_flush<true>(f, A, sm.stage, sm.edge_s, hist2);
    {
      const OpUnit A2 = op_decode(f, tA2);
      pv = load_partial_coherent(f.bias + (int64_t)A2.seg * a.row_slots +
                                 min(tid, max(A2.rt_n, 1) * 16 - 1));
    }
    // 5. B's statistics, published; the arrival and the next ticket
    if (B.valid) {
      const float2 mine = op_unit_stats<RTM>(a, B, ev[P], mu_s[P], part);
      if (tid < B.rt_n * 16)
        store_partial_coherent(op_partials(a, B) + (int64_t)B.u * a.row_slots + tid,
                               make_float2(mine.x, -mine.y));
      t_pub = tB;
    }
    __syncthreads();   // every partial store is issued before the arrival
    if (tid == 0) {
      if (t_pub >= 0)
        arrived = __hip_atomic_fetch_add(&f.arrive[B.seg], 1, __ATOMIC_RELAXED,
                                         __HIP_MEMORY_SCOPE_AGENT);
      tk_req = atomicAdd(f.ticket, 1);
    }
    // 6. unit k + 1's loads into the registers B's operands came from (after
    //    the atomics, so that reading their results does not wait for them)
    op_unit_loads<T, D, RTM>(a, op_decode(f, tC), kr, qv);
    tA = tA2;
    tA2 = tB;
    tB = tC;
    auto live = [&](int t) { return t >= 0 && t < f.n_units_total; };
    return live(tA) || live(tA2) || live(tB);
  };
  for (;;) {
    if (!iterate.template operator()<0>()) break;
    if (!iterate.template operator()<1>()) break;
  }
}

// Units whose normalisers had not arrived when the main kernel reached them:
// the segment's normalisers are merged here from the (now complete) unit
// partials, the unit's statistics are recomputed from its keys, and it is
// finished, all with the main kernel's code and order of operations.
template <typename T, int D, int RTM>
__global__ __launch_bounds__(kOpThreads) void onepass_catchup_kernel(const OnePassArgs f) {
  constexpr int NS = Slices<T, D>::n;
  constexpr int QN = QStage<T, D, RTM, kOpThreads>::n;
  const ScoreArgs &a = f.s;
  __shared__ OpLds<T, D, RTM, 1> sm;
  uint4 *q_lds = sm.q[0];
  auto &part = sm.u.part;
  auto &cs = sm.u.cs;
  float *bias_s = sm.bias_s;
  float *mu_s = sm.mu_s[0];
  uint32_t *hist2 = sm.hist2;
  for (int i = threadIdx.x; i < kHistBins / 2; i += kOpThreads) hist2[i] = 0;
  const int n = *f.skip_count;
  for (int i = blockIdx.x; i < n; i += gridDim.x) {
    const OpUnit x = op_decode(f, f.skip_list[i]);
    if (!x.valid) continue;
    uint4 kr[kOpTiles][NS];
    uint4 qv[QN];
    f32x4 e[kOpTiles][RTM];
    op_unit_loads<T, D, RTM>(a, x, kr, qv);
    __syncthreads();   // q_lds and bias_s of the previous unit are no longer read
    q_store<T, D, RTM, kOpThreads>(qv, q_lds);
    op_merge_segment(a, x, 0, RTM * 16, bias_s);   // ends with a barrier
    op_unit_logits<T, D, RTM>(x, kr, q_lds, e);
    op_unit_stats<RTM>(a, x, e, mu_s, part);
    op_unit_finish<RTM>(f, x, e, mu_s, bias_s, cs, sm.stage, sm.edge_s, hist2);
    op_unit_flush<false>(f, x, sm.stage, sm.edge_s, hist2);
  }
}

// Positions within r of a boundary between units u - 1 and u of a segment
// (u >= 1, boundary u0 = 256 u < P): pooled from the window sums both units
// stored at their ends, one thread per position.
__global__ __launch_bounds__(256) void onepass_boundary_kernel(const OnePassArgs f) {
  const ScoreArgs &a = f.s;
  const int ew = f.ew, rp = ew / 2;
  const int64_t gid = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (ew == 0 || gid >= (int64_t)f.n_units_total * ew) return;
  const int ticket = (int)(gid / ew), o = (int)(gid % ew);
  const OpUnit x = op_decode<false>(f, ticket);
  if (!x.valid || x.u == 0 || x.u0 >= x.P) return;
  const int pos = x.u0 - rp + o;
  if (pos >= x.P) return;
  const int hs = f.heads_max * 2 * ew;
  const float *right = f.edges + (int64_t)ticket * hs;        // unit u: side 0
  const float *left = f.edges + (int64_t)(ticket - 1) * hs;   // unit u - 1: side 1
  auto cs_at = [&](int h, int p) {
    return p >= x.u0 ? right[(h * 2 + 0) * ew + (p - x.u0)]
                     : left[(h * 2 + 1) * ew + (p - (x.u0 - ew))];
  };
  const float score = op_pool(a, cs_at, x.nh, pos, x.P);
  const LayerView lv = layer_view<true>(a, x.layer, x.g);
  lv.scores[(int64_t)x.g * a.T + x.s0 + pos] = score;
  atomicAdd(a.hist + x.layer * a.hist_layer + (int64_t)x.gi * kHistBins +
                hist_bin(__float_as_uint(score)),
            1);
}

// ---------------------------------------------------------------------------
// Host side
// ---------------------------------------------------------------------------
template <typename T, int D, int RTM>
static hipError_t launch_onepass_t(const OnePassArgs &f, int grid, int64_t fill_ints,
                                   hipStream_t stream) {
  hipLaunchKernelGGL(op_fill_kernel, dim3(1024), dim3(256), 0, stream, f.fill_base, fill_ints);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((onepass_kernel<T, D, RTM>), dim3(grid), dim3(kOpThreads), 0, stream, f);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL((onepass_catchup_kernel<T, D, RTM>), dim3(grid), dim3(kOpThreads), 0,
                     stream, f);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (f.ew > 0) {
    const int64_t n = (int64_t)f.n_units_total * f.ew;
    hipLaunchKernelGGL(onepass_boundary_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0,
                       stream, f);
    e = hipGetLastError();
  }
  return e;
}

// One instance per head size: its body skips the row tiles a group does not
// have (uniform branches), so it serves every group of up to 6 row tiles.
constexpr int kOpRowTiles = 6;

hipError_t launch_onepass(const OnePassArgs &f, int head_dim, int rt_max, int grid,
                          int64_t fill_ints, hipStream_t stream) {
  if (grid < 1 || f.n_units_total < 1 || rt_max > kOpRowTiles)
    return hipErrorInvalidConfiguration;
  return head_dim == 64
             ? launch_onepass_t<__bf16, 64, kOpRowTiles>(f, grid, fill_ints, stream)
             : launch_onepass_t<__bf16, 128, kOpRowTiles>(f, grid, fill_ints, stream);
}

}  // namespace ckv
