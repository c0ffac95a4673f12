// S5 keeps, per (sequence, KV group), the (budget - W) highest prefix scores
// (section 3.3: the N best tokens keep their KV pairs) with ties going to the
// lowest position, plus the W window positions, written in ascending order.
// Scores are non-negative floats, so their bit patterns order like unsigned
// integers.  A three-digit radix select finds the exact bit pattern of the
// k-th largest score: digit 1 (bits 30..20) comes from the histogram that the
// column-sum kernel accumulated (or is counted here), the elements of the
// chosen bucket are collected in LDS, and digits 2 (bits 19..9) and 3 (bits
// 8..0) are resolved on that candidate list.  An ordered compaction then
// writes the kept positions.  Integer work only, so the result does not
// depend on scheduling.  Every wave holds a contiguous run of positions with
// its lanes on neighbouring positions, so the score loads are coalesced and
// the compaction orders kept positions with wave ballots.
//
// S6 copies the kept K and V rows (section 3.3: the retained KV pairs form the
// compressed cache) with 16-byte lanes; rows whose index is -1 become zeros.
//
// ML (multi-layer): the grid's last dimension runs over (layer, sequence)
// pairs, layer-major, and each layer's operands and budget come from the table.
#include "ckv_launch.h"

namespace ckv {

constexpr int kSelThreads = 1024;
constexpr int kCandCap = 8192;               // candidates of the first-digit bucket kept in LDS
// Scores per thread held in registers per round: the split selection's
// slices are one round of kEpt; a whole selection in one workgroup uses
// kEptWhole (fewer registers held across all its passes).
constexpr int kEpt = 32;
constexpr int kRound = kSelThreads * kEpt;
static_assert(kRound == kSelSlice, "a slice of the split selection is one round");
constexpr int kEptWhole = 16;
constexpr int kRoundWhole = kSelThreads * kEptWhole;

// Inclusive prefix sum over the 1024 threads of the block; *total gets the sum.
__device__ __forceinline__ int block_inclusive_scan(int x, int *lds_waves, int *total) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    int y = __shfl_up(x, o);
    if (lane >= o) x += y;
  }
  if (lane == 63) lds_waves[wave] = x;
  __syncthreads();
  if (wave == 0) {
    int w = (lane < kSelThreads / 64) ? lds_waves[lane] : 0;
#pragma unroll
    for (int o = 1; o < 16; o <<= 1) {
      int y = __shfl_up(w, o);
      if (lane >= o) w += y;
    }
    if (lane < kSelThreads / 64) lds_waves[lane] = w;
  }
  __syncthreads();
  const int before = (wave > 0) ? lds_waves[wave - 1] : 0;
  *total = lds_waves[kSelThreads / 64 - 1];
  __syncthreads();   // lds_waves is reused by the next scan
  return x + before;
}

// LDS histogram increment; a wave whose active lanes share one bin issues a
// single atomic (plateaus of equal scores are common after max pooling).
// Must be reached by every lane of the wave.
__device__ __forceinline__ void hist_add(int *h, int bin, bool active) {
  const unsigned long long m = __ballot(active);
  if (m == 0ull) return;
  const int leader = __ffsll((unsigned long long)m) - 1;
  const int first = __shfl(bin, leader);
  if (__all(!active || bin == first)) {
    if ((int)(threadIdx.x & 63) == leader) atomicAdd(&h[first], (int)__popcll(m));
  } else if (active) {
    atomicAdd(&h[bin], 1);
  }
}

// Bucket of an nb-bin histogram (nb <= 2048) that holds the element of rank
// `remain` counted from the top; writes the bucket and the rank inside it.
__device__ __forceinline__ void find_bucket(const int *hist, int nb, int remain, int *scan_tmp,
                                            int *bucket_out, int *remain_out) {
  const int tid = threadIdx.x;
  const int hi_b = nb - 1 - 2 * tid;     // thread t owns buckets nb-1-2t and nb-2-2t
  const int c_hi = (hi_b >= 0) ? hist[hi_b] : 0;
  const int c_lo = (hi_b - 1 >= 0) ? hist[hi_b - 1] : 0;
  int total;
  const int incl = block_inclusive_scan(c_hi + c_lo, scan_tmp, &total);
  const int excl = incl - c_hi - c_lo;   // elements in buckets above hi_b
  if (hi_b >= 0) {
    if (excl < remain && remain <= excl + c_hi) {
      *bucket_out = hi_b;
      *remain_out = remain - excl;
    } else if (hi_b - 1 >= 0 && excl + c_hi < remain && remain <= excl + c_hi + c_lo) {
      *bucket_out = hi_b - 1;
      *remain_out = remain - excl - c_hi;
    }
  }
  __syncthreads();
}

// Position of a thread's element e in the round starting at r0: every wave
// owns a run of 64 * EPT consecutive positions and its lanes take
// consecutive positions for each e, so a load instruction reads 256
// contiguous bytes and the position order is (wave, e, lane).
template <int EPT>
__device__ __forceinline__ int elem_pos(int r0, int e) {
  return r0 + (int)(threadIdx.x >> 6) * (64 * EPT) + e * 64 + (int)(threadIdx.x & 63);
}

// Lanes below this one whose bit is set in m.
__device__ __forceinline__ int lanes_below(unsigned long long m) {
  return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                        __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

// A thread's EPT scores of the round starting at r0 into registers, all
// loads issued together.  They go through a buffer resource whose range is
// the P prefix scores, so positions >= P read as 0 without a branch or a
// clamp (the callers mask them).
template <int EPT>
__device__ __forceinline__ void load_round(gptr<const uint32_t> sc, int P, int r0,
                                           uint32_t (&v)[EPT]) {
  // raw buffer (stride 0), 32-bit data format; range P * 4 bytes
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
      (void *)sc, (short)0, P * 4, 0x00020000);
  const int off = elem_pos<EPT>(r0, 0) * 4;
#pragma unroll
  for (int e = 0; e < EPT; ++e) v[e] = __builtin_amdgcn_raw_buffer_load_b32(rs, off + e * 256, 0, 0);
}

// One selection: (layer, sequence b, selection index g) with its operands.
struct Sel {
  LayerView lv;
  int layer, b, g, budget, L, P, k;
  int64_t id;                    // (layer * batch + b) * n_sel + g
  gptr<int32_t> out;             // the kept list of (b, g)
  gptr<const uint32_t> sc;       // the selection's scores, position 0 of the sequence
};

// lb = layer * batch + b.
template <bool ML>
__device__ __forceinline__ Sel sel_of(const SelectArgs &a, int g, int lb) {
  Sel s;
  s.g = g;
  s.layer = ML ? lb / a.batch : 0;
  s.b = lb - s.layer * a.batch;
  s.lv = layer_view<ML>(a, s.layer, 0);
  s.budget = a.gb.on ? a.gb.budget[g] : s.lv.budget;
  const int s0 = a.cu[s.b];
  s.L = a.cu[s.b + 1] - s0;
  s.P = s.L - a.W;
  s.k = s.budget - a.W;           // prefix tokens to keep when L > budget: 0 <= k < P
  s.id = (int64_t)lb * a.n_sel + g;
  s.out = s.lv.idx + kept_base(a.gb, s.b, g, a.Hkv, s.budget);
  s.sc = reinterpret_cast<gptr<const uint32_t>>(s.lv.scores + (int64_t)g * a.T + s0);
  return s;
}

// Position `pos` of the kept list, in every idx row this selection serves.
__device__ __forceinline__ void sel_put(const SelectArgs &a, const Sel &s, int pos, int32_t val) {
  for (int r = 0; r < a.out_groups; ++r) s.out[(int64_t)r * s.budget + pos] = val;
}

// The part of the kept list that needs no selection: everything when
// L <= budget (slots past L get -1), else the window positions.  True when
// nothing is left to select.
__device__ __forceinline__ bool sel_trivial(const SelectArgs &a, const Sel &s) {
  const int tid = threadIdx.x;
  if (s.L <= s.budget) {
    for (int j = tid; j < s.budget; j += kSelThreads) sel_put(a, s, j, (j < s.L) ? j : -1);
    return true;
  }
  for (int w = tid; w < a.W; w += kSelThreads) sel_put(a, s, s.k + w, s.P + w);
  return s.k == 0;
}

// The first-digit histogram of a selection into LDS: from the column-sum
// kernel's, or counted over the prefix scores.
__device__ __forceinline__ void sel_hist1(const SelectArgs &a, const Sel &s, int *hist,
                                          uint32_t (&v)[kEptWhole], bool resident, int nrounds) {
  const int tid = threadIdx.x;
  if (a.hist) {
    const int *hg = a.hist + s.layer * a.hist_layer + ((int64_t)s.b * a.Hkv + s.g) * kHistBins;
    for (int i = tid; i < kHistBins; i += kSelThreads) hist[i] = hg[i];
    return;
  }
  for (int i = tid; i < kHistBins; i += kSelThreads) hist[i] = 0;
  __syncthreads();
  for (int r = 0; r < nrounds; ++r) {
    if (!resident) load_round(s.sc, s.P, r * kRoundWhole, v);
#pragma unroll
    for (int e = 0; e < kEptWhole; ++e)
      hist_add(hist, hist_bin(v[e]), elem_pos<kEptWhole>(r * kRoundWhole, e) < s.P);
  }
}

// Slot of this lane in a list that the wave appends its flagged lanes to
// (one LDS atomic per wave); every lane of the wave must reach it.
__device__ __forceinline__ int wave_append(int *count, bool flag) {
  const unsigned long long m = __ballot(flag);
  if (m == 0ull) return 0;
  const int leader = __ffsll((unsigned long long)m) - 1;
  int base = 0;
  if ((int)(threadIdx.x & 63) == leader) base = atomicAdd(count, (int)__popcll(m));
  base = __shfl(base, leader);
  return base + lanes_below(m);
}

// Ordered compaction of the round starting at r0 (this thread's scores in v):
// keeps the elements above thr and, of those equal to it, the ones whose rank
// among the sequence's ties (eq_base ties come before this round) is below
// `remain`; writes them from kept-list position pos_base on, in position
// order.  Each wave counts its elements above and at the threshold, every
// wave forms the prefix over the waves before it, and the kept positions are
// written in (wave, e, lane) order.  Returns the kept count through *kept
// and the tie count through *ties.
template <int EPT>
__device__ __forceinline__ void compact_round(const SelectArgs &a, const Sel &s,
                                              const uint32_t (&v)[EPT], int r0, uint32_t thr,
                                              int remain, int pos_base, int eq_base,
                                              int (*wave_cnt)[kSelThreads / 64], int *kept,
                                              int *ties) {
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  int n_gt = 0, n_eq = 0;   // this thread's counts, then the wave's
#pragma unroll
  for (int e = 0; e < EPT; ++e) {
    const uint32_t u = v[e] & 0x7FFFFFFFu;
    const bool ok = elem_pos<EPT>(r0, e) < s.P;
    n_gt += ok && u > thr;
    n_eq += ok && u == thr;
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) {
    n_gt += __shfl_xor(n_gt, o);
    n_eq += __shfl_xor(n_eq, o);
  }
  if (lane == 0) {
    wave_cnt[0][wave] = n_gt;
    wave_cnt[1][wave] = n_eq;
  }
  __syncthreads();
  int eq_before = 0, sel_before = 0, eq_total = 0, sel_total = 0;
#pragma unroll
  for (int x = 0; x < kSelThreads / 64; ++x) {
    const int c_gt = wave_cnt[0][x], c_eq = wave_cnt[1][x];
    const int take = max(0, min(c_eq, remain - (eq_base + eq_total)));   // wave x's kept ties
    if (x < wave) {
      eq_before += c_eq;
      sel_before += c_gt + take;
    }
    eq_total += c_eq;
    sel_total += c_gt + take;
  }
  __syncthreads();   // wave_cnt is rewritten by the next round
  int pos = pos_base + sel_before;
  int eq_rank = eq_base + eq_before;
#pragma unroll
  for (int e = 0; e < EPT; ++e) {
    const int j = elem_pos<EPT>(r0, e);
    const uint32_t u = v[e] & 0x7FFFFFFFu;
    const bool ok = j < s.P;
    const bool gt = ok && u > thr, eq = ok && u == thr;
    const unsigned long long m_gt = __ballot(gt), m_eq = __ballot(eq);
    if ((m_gt | m_eq) == 0ull) continue;   // nothing kept at this e (uniform; most e)
    const bool keep = gt || (eq && eq_rank + lanes_below(m_eq) < remain);
    const unsigned long long m_keep = __ballot(keep);
    const int my_pos = pos + lanes_below(m_keep);
    if (keep && my_pos < s.k) sel_put(a, s, my_pos, j);   // bound holds for finite scores; guards NaN
    pos += __popcll(m_keep);
    eq_rank += __popcll(m_eq);
  }
  *kept = sel_total;
  *ties = eq_total;
}

struct SelLds {
  int hist[kHistBins];
  int scan_tmp[kSelThreads / 64];
  int wave_cnt[2][kSelThreads / 64];
  int bucket, remain, ncand;
  uint32_t cand_u[kCandCap];
};

// The whole selection in one workgroup (after sel_trivial): digit 1 from the
// histogram, the elements of its bucket collected in LDS, digits 2 (bits
// 19..9) and 3 (bits 8..0) on that list (or, if it overflows, on every
// prefix element that matches so far), then the ordered compaction, round by
// round.
__device__ __forceinline__ void select_whole(const SelectArgs &a, const Sel &s, SelLds &lds) {
  const int tid = threadIdx.x;
  const int nrounds = (s.P + kRoundWhole - 1) / kRoundWhole;
  const bool resident = (nrounds == 1);   // scores stay in registers for every pass
  uint32_t v[kEptWhole];
  if (resident) load_round(s.sc, s.P, 0, v);
  sel_hist1(a, s, lds.hist, v, resident, nrounds);
  if (tid == 0) {
    lds.ncand = 0;
    lds.bucket = 0;
    lds.remain = 0;
  }
  __syncthreads();
  find_bucket(lds.hist, kHistBins, s.k, lds.scan_tmp, &lds.bucket, &lds.remain);
  uint32_t pmask = 0x7FFu << 20;
  uint32_t prefix = (uint32_t)lds.bucket << 20;
  int remain = lds.remain;

  for (int r = 0; r < nrounds; ++r) {
    if (!resident) load_round(s.sc, s.P, r * kRoundWhole, v);
#pragma unroll
    for (int e = 0; e < kEptWhole; ++e) {
      const bool c = elem_pos<kEptWhole>(r * kRoundWhole, e) < s.P && (v[e] & pmask) == prefix;
      const int slot = wave_append(&lds.ncand, c);
      if (c && slot < kCandCap) lds.cand_u[slot] = v[e];
    }
  }
  __syncthreads();
  const int nc = lds.ncand;
  const bool in_lds = nc <= kCandCap;

  const int shifts[2] = {9, 0};
  const int widths[2] = {11, 9};
  for (int pass = 0; pass < 2; ++pass) {
    const int sh = shifts[pass];
    const uint32_t dmask = (1u << widths[pass]) - 1u;
    for (int i = tid; i < kHistBins; i += kSelThreads) lds.hist[i] = 0;
    __syncthreads();
    if (in_lds) {
      for (int base = 0; base < nc; base += kSelThreads) {
        const int i = base + tid;
        const uint32_t u = (i < nc) ? lds.cand_u[i] : 0u;
        hist_add(lds.hist, (int)((u >> sh) & dmask), i < nc && (u & pmask) == prefix);
      }
    } else {
      for (int r = 0; r < nrounds; ++r) {
        if (!resident) load_round(s.sc, s.P, r * kRoundWhole, v);
#pragma unroll
        for (int e = 0; e < kEptWhole; ++e)
          hist_add(lds.hist, (int)((v[e] >> sh) & dmask),
                   elem_pos<kEptWhole>(r * kRoundWhole, e) < s.P && (v[e] & pmask) == prefix);
      }
    }
    __syncthreads();
    find_bucket(lds.hist, 1 << widths[pass], remain, lds.scan_tmp, &lds.bucket, &lds.remain);
    prefix |= (uint32_t)lds.bucket << sh;
    pmask |= dmask << sh;
    remain = lds.remain;
    __syncthreads();
  }

  // prefix is the exact bit pattern of the k-th largest score; `remain` of
  // the positions holding it are kept (the lowest ones), plus every larger
  // score.
  int pos_base = 0, eq_base = 0;
  for (int r = 0; r < nrounds; ++r) {
    if (!resident) load_round(s.sc, s.P, r * kRoundWhole, v);
    int kept, ties;
    compact_round(a, s, v, r * kRoundWhole, prefix, remain, pos_base, eq_base, lds.wave_cnt, &kept,
                  &ties);
    pos_base += kept;
    eq_base += ties;
  }
}

// Grid (n_sel, batch [x layers]), 1024 threads: one selection per workgroup.
template <bool ML>
__global__ __launch_bounds__(kSelThreads) void select_kernel(const SelectArgs a) {
  const Sel s = sel_of<ML>(a, blockIdx.x, blockIdx.y);
  if (sel_trivial(a, s)) return;
  __shared__ SelLds lds;
  select_whole(a, s, lds);
}

// Long sequences: the selection split over its rounds ("slices" of kRound
// positions), in three launches with the same result as select_kernel.
//  scan:    per slice, the elements of the first-digit bucket (its
//           candidates) into the slice's candidate list, and every element
//           at or above the bucket, as a (position, score) pair, into the
//           wave's part of the slice's ordered list (ascending positions);
//           slice 0 also passes the first digit on;
//  resolve: per selection, digits 2 and 3 over all the slices' candidates,
//           then each slice's first kept-list position and ties before it;
//  write:   per slice, the ordered compaction of its ordered list.
static_assert(kSelMetaPerSlice == 1 + kSelThreads / 64 + 4, "meta words of a slice");
constexpr int kMetaFirst = 1 + kSelThreads / 64;   // first kept-list position
constexpr int kMetaTies = kMetaFirst + 1;           // ties in the slices before
// The last two words: the threshold (score bits) and the ties kept in all,
// from the resolve kernel; before it, slice 0's hold the first-digit bucket
// and the rank inside it, from the scan.
constexpr int kMetaThr = kMetaFirst + 2;
constexpr int kMetaRemain = kMetaFirst + 3;

__device__ __forceinline__ int *sel_meta(const SelectArgs &a, const Sel &s) {
  return a.sel_meta + s.id * (kSelMetaPerSlice * a.n_slices);
}

// Grid (n_slices, n_sel, batch [x layers]), 1024 threads.
template <bool ML>
__global__ __launch_bounds__(kSelThreads) void select_scan_kernel(const SelectArgs a) {
  const Sel s = sel_of<ML>(a, blockIdx.y, blockIdx.z);
  const int slice = blockIdx.x;
  const int r0 = slice * kRound;
  if (s.L <= s.budget || s.k == 0 || r0 >= s.P) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  __shared__ int hist[kHistBins];
  __shared__ int scan_tmp[kSelThreads / 64];
  __shared__ int bucket_s, remain_s, ncand_s;
  uint32_t v[kEpt];
  load_round(s.sc, s.P, r0, v);
  const int *hg = a.hist + s.layer * a.hist_layer + ((int64_t)s.b * a.Hkv + s.g) * kHistBins;
  for (int i = tid; i < kHistBins; i += kSelThreads) hist[i] = hg[i];
  if (tid == 0) {
    bucket_s = 0;
    remain_s = 0;
    ncand_s = 0;
  }
  __syncthreads();
  find_bucket(hist, kHistBins, s.k, scan_tmp, &bucket_s, &remain_s);
  const int bucket = bucket_s;
  if (slice == 0 && tid == 0) {   // the same in every slice: for the resolve kernel
    int *meta0 = sel_meta(a, s);
    meta0[kMetaThr] = bucket;
    meta0[kMetaRemain] = remain_s;
  }
  // The bucket's elements go to the candidate list in no particular order
  // (the resolve kernel only counts them); the elements at or above it go to
  // the wave's part of the ordered list (its 64 * kEpt positions, in (e,
  // lane) order, i.e. ascending), bit 31 of the position marking a candidate.
  const int64_t list = (s.id * a.n_slices + slice) * (int64_t)a.cand_cap;
  const gptr<uint32_t> cand = to_global(a.sel_cand) + list;
  const gptr<uint64_t> ord = to_global(a.sel_ord) + list + wave * (64 * kEpt);
  // the wave's candidates are counted first, so that one LDS atomic
  // reserves their slots
  int n_cand = 0;
#pragma unroll
  for (int e = 0; e < kEpt; ++e)
    n_cand += (int)__popcll(__ballot(elem_pos<kEpt>(r0, e) < s.P && hist_bin(v[e]) == bucket));
  // (the scores are recomputed from below, not kept from the count)
  int j0 = elem_pos<kEpt>(r0, 0);
#pragma unroll
  for (int e = 0; e < kEpt; ++e) asm volatile("" : "+v"(v[e]));
  asm volatile("" : "+v"(j0));
  int cand_at = 0;
  if (lane == 0 && n_cand) cand_at = atomicAdd(&ncand_s, n_cand);
  cand_at = __shfl(cand_at, 0);
  int n_ord = 0;
#pragma unroll
  for (int e = 0; e < kEpt; ++e) {
    const int j = j0 + 64 * e;   // elem_pos<kEpt>(r0, e)
    const bool ok = j < s.P;
    const int bin = hist_bin(v[e]);
    const bool c = ok && bin == bucket;
    const unsigned long long m_c = __ballot(c);
    if (c && cand_at + lanes_below(m_c) < a.cand_cap) cand[cand_at + lanes_below(m_c)] = v[e];
    cand_at += (int)__popcll(m_c);
    const bool f = ok && bin >= bucket;
    const unsigned long long m = __ballot(f);
    if (f)
      ord[n_ord + lanes_below(m)] = ((uint64_t)(v[e] & 0x7FFFFFFFu) << 32) |
                                    (uint32_t)j | (c ? 0x80000000u : 0u);
    n_ord += (int)__popcll(m);
    __builtin_amdgcn_sched_barrier(0);   // one element's stores at a time
  }
  int *meta = sel_meta(a, s) + slice * kSelMetaPerSlice;
  if ((tid & 63) == 0) meta[1 + wave] = n_ord;
  __syncthreads();
  if (tid == 0) meta[0] = ncand_s;
}

// Candidates the resolve kernel keeps in LDS (32 KB), loaded kResolveEpt
// per thread at a time; more are read from the slices' lists on every pass.
constexpr int kResolveCandCap = 8192;
constexpr int kResolveEpt = 8;

struct ResolveLds {
  int hist[kHistBins];
  int scan_tmp[kSelThreads / 64];
  int bucket, remain;
  int cand_off[kMaxSelSlices + 1], above[kMaxSelSlices], gt[kMaxSelSlices], eq[kMaxSelSlices];
  uint32_t cand_u[kResolveCandCap];
};

// Grid (n_sel, batch [x layers]), 1024 threads.
template <bool ML>
__global__ __launch_bounds__(kSelThreads) void select_resolve_kernel(const SelectArgs a) {
  const Sel s = sel_of<ML>(a, blockIdx.x, blockIdx.y);
  const int tid = threadIdx.x;
  if (sel_trivial(a, s)) return;
  int *meta = sel_meta(a, s);
  __shared__ ResolveLds lds;
  const int ns = (s.P + kRound - 1) / kRound;
  const int nsl = a.n_slices;
  if (tid == 0) {   // digit 1, found by the scan
    lds.bucket = meta[kMetaThr];
    lds.remain = meta[kMetaRemain];
  }
  if (tid < ns) {
    const int *m = meta + tid * kSelMetaPerSlice;
    int n_ord = 0;
    for (int w = 0; w < kSelThreads / 64; ++w) n_ord += m[1 + w];
    lds.cand_off[tid + 1] = m[0];          // <= cand_cap: a slice's positions
    lds.above[tid] = n_ord - m[0];         // the list holds the candidates and those above
    lds.gt[tid] = 0;
    lds.eq[tid] = 0;
  }
  __syncthreads();
  if (tid == 0) {
    lds.cand_off[0] = 0;
    for (int sl = 0; sl < ns; ++sl) lds.cand_off[sl + 1] += lds.cand_off[sl];
  }
  __syncthreads();
  uint32_t prefix = (uint32_t)lds.bucket << 20;
  int remain = lds.remain;
  const int nc = lds.cand_off[ns];
  const gptr<const uint32_t> cand0 = to_global(a.sel_cand) + s.id * nsl * (int64_t)a.cand_cap;
  // Candidate i of the concatenation (slices in order) lies in slice sl
  // (cand_off[sl] <= i < cand_off[sl + 1]).  Into LDS kResolveEpt per thread
  // at a time: addresses first, then every load at once.
  const bool in_lds = nc <= kResolveCandCap;
  if (in_lds) {
    int sl = 0;
    for (int base = 0; base < nc; base += kResolveEpt * kSelThreads) {
      int64_t at[kResolveEpt];
#pragma unroll
      for (int m = 0; m < kResolveEpt; ++m) {
        const int i = base + m * kSelThreads + tid;
        at[m] = 0;   // past the end: a valid address, not stored
        if (i < nc) {
          while (lds.cand_off[sl + 1] <= i) ++sl;
          at[m] = sl * (int64_t)a.cand_cap + (i - lds.cand_off[sl]);
        }
      }
      uint32_t u[kResolveEpt];
#pragma unroll
      for (int m = 0; m < kResolveEpt; ++m) u[m] = cand0[at[m]];
#pragma unroll
      for (int m = 0; m < kResolveEpt; ++m)
        if (base + m * kSelThreads + tid < nc) lds.cand_u[base + m * kSelThreads + tid] = u[m];
    }
  }
  // fn(u, slice, valid) over every candidate, slice by slice; every thread
  // makes the same calls.
  auto each = [&](auto fn) {
    for (int sl = 0; sl < ns; ++sl) {
      const int c0 = lds.cand_off[sl], n = lds.cand_off[sl + 1] - c0;
      if (in_lds) {
        for (int base = 0; base < n; base += kSelThreads) {
          const int i = base + tid;
          fn(i < n ? lds.cand_u[c0 + i] : 0u, sl, i < n);
        }
      } else {
        const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
            (void *)(cand0 + sl * (int64_t)a.cand_cap), (short)0, n * 4, 0x00020000);
        for (int base = 0; base < n; base += kResolveEpt * kSelThreads) {
          uint32_t u[kResolveEpt];
#pragma unroll
          for (int m = 0; m < kResolveEpt; ++m)
            u[m] = __builtin_amdgcn_raw_buffer_load_b32(rs, (base + m * kSelThreads + tid) * 4,
                                                        0, 0);
#pragma unroll
          for (int m = 0; m < kResolveEpt; ++m) fn(u[m], sl, base + m * kSelThreads + tid < n);
        }
      }
    }
  };
  __syncthreads();
  // digits 2 (bits 19..9) and 3 (bits 8..0) over the candidates
  const int shifts[2] = {9, 0};
  const int widths[2] = {11, 9};
  uint32_t pmask = 0x7FFu << 20;
  for (int pass = 0; pass < 2; ++pass) {
    const int sh = shifts[pass];
    const uint32_t dmask = (1u << widths[pass]) - 1u;
    for (int i = tid; i < kHistBins; i += kSelThreads) lds.hist[i] = 0;
    __syncthreads();
    each([&](uint32_t u, int, bool ok) {
      hist_add(lds.hist, (int)((u >> sh) & dmask), ok && (u & pmask) == prefix);
    });
    __syncthreads();
    find_bucket(lds.hist, 1 << widths[pass], remain, lds.scan_tmp, &lds.bucket, &lds.remain);
    prefix |= (uint32_t)lds.bucket << sh;
    pmask |= dmask << sh;
    remain = lds.remain;
    __syncthreads();
  }
  const uint32_t thr = prefix;
  // per slice: candidates above the threshold (added to the slice's elements
  // above the bucket) and ties
  each([&](uint32_t u, int sl, bool ok) {
    const uint32_t x = u & 0x7FFFFFFFu;
    const int n_gt = (int)__popcll(__ballot(ok && x > thr));
    const int n_eq = (int)__popcll(__ballot(ok && x == thr));
    if ((threadIdx.x & 63) == 0) {
      if (n_gt) atomicAdd(&lds.gt[sl], n_gt);
      if (n_eq) atomicAdd(&lds.eq[sl], n_eq);
    }
  });
  __syncthreads();
  if (tid == 0) {
    int pos = 0, ties = 0;
    for (int sl = 0; sl < ns; ++sl) {
      int *m = meta + sl * kSelMetaPerSlice;
      m[kMetaFirst] = pos;
      m[kMetaTies] = ties;
      m[kMetaThr] = (int)thr;
      m[kMetaRemain] = remain;
      const int gt = lds.above[sl] + lds.gt[sl];
      pos += gt + max(0, min(lds.eq[sl], remain - ties));
      ties += lds.eq[sl];
    }
  }
}

// Ordered-list entries per lane per batch of the write kernel.
constexpr int kWriteEpt = 8;
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// Grid (n_slices, n_sel, batch [x layers]), 1024 threads.  Wave w compacts
// the slice's ordered-list part w (ascending positions, 64 entries per
// step), reading it twice: it counts its entries above the threshold and its ties, the waves'
// counts are exchanged, and it writes its kept positions from the slice's
// first kept-list position on.  An entry above the threshold is kept, and of
// those equal to it the first `remain` of the sequence in position order.
template <bool ML>
__global__ __launch_bounds__(kSelThreads) void select_write_kernel(const SelectArgs a) {
  const Sel s = sel_of<ML>(a, blockIdx.y, blockIdx.z);
  const int slice = blockIdx.x;
  const int r0 = slice * kRound;
  if (s.L <= s.budget || s.k == 0 || r0 >= s.P) return;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  __shared__ int wave_cnt[2][kSelThreads / 64];
  const int *meta = sel_meta(a, s) + slice * kSelMetaPerSlice;
  const int n = meta[1 + wave];
  const uint32_t thr = (uint32_t)meta[kMetaThr];
  const int room = max(0, meta[kMetaRemain] - meta[kMetaTies]);   // ties still to keep
  // the wave's part through a buffer resource of n entries: loads past the
  // end read 0 (and are masked below)
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
      (void *)(a.sel_ord + (s.id * a.n_slices + slice) * (int64_t)a.cand_cap +
               wave * (64 * kEpt)),
      (short)0, n * 8, 0x00020000);
  auto above = [&](const uint64_t x, bool valid) {
    return valid && ((((uint32_t)x >> 31) == 0u) || (uint32_t)(x >> 32) > thr);
  };
  auto equal = [&](const uint64_t x, bool valid) {
    return valid && ((uint32_t)x >> 31) != 0u && (uint32_t)(x >> 32) == thr;
  };
  // kWriteEpt entries per lane at a time, every load of a batch at once
  auto load = [&](int b, uint64_t (&e)[kWriteEpt]) {
#pragma unroll
    for (int m = 0; m < kWriteEpt; ++m) {
      const u32x2 r = __builtin_amdgcn_raw_buffer_load_b64(rs, (b + 64 * m + lane) * 8, 0, 0);
      e[m] = ((uint64_t)r.y << 32) | r.x;
    }
  };
  int c_gt = 0, c_eq = 0;
  for (int b = 0; b < n; b += 64 * kWriteEpt) {
    uint64_t e[kWriteEpt];
    load(b, e);
#pragma unroll
    for (int m = 0; m < kWriteEpt; ++m) {
      const bool valid = b + 64 * m + lane < n;
      c_gt += (int)__popcll(__ballot(above(e[m], valid)));
      c_eq += (int)__popcll(__ballot(equal(e[m], valid)));
    }
  }
  if (lane == 0) {
    wave_cnt[0][wave] = c_gt;
    wave_cnt[1][wave] = c_eq;
  }
  __syncthreads();
  int gt_before = 0, eq_before = 0;
#pragma unroll
  for (int x = 0; x < kSelThreads / 64; ++x) {
    if (x < wave) {
      gt_before += wave_cnt[0][x];
      eq_before += wave_cnt[1][x];
    }
  }
  int my = meta[kMetaFirst] + gt_before + min(eq_before, room);
  int eq_rank = eq_before;
  for (int b = 0; b < n; b += 64 * kWriteEpt) {
    uint64_t e[kWriteEpt];
    load(b, e);
#pragma unroll
    for (int m = 0; m < kWriteEpt; ++m) {
      const bool valid = b + 64 * m + lane < n;
      const bool eq = equal(e[m], valid);
      const unsigned long long m_eq = __ballot(eq);
      const bool keep = above(e[m], valid) || (eq && eq_rank + lanes_below(m_eq) < room);
      const unsigned long long m_keep = __ballot(keep);
      const int slot = my + lanes_below(m_keep);
      if (keep && slot < s.k) sel_put(a, s, slot, (int)((uint32_t)e[m] & 0x7FFFFFFFu));
      my += (int)__popcll(m_keep);
      eq_rank += (int)__popcll(m_eq);
    }
  }
}

// Grid (ceil(max budget / rows_per_block), Hkv, batch [x layers]), 256
// threads; each lane moves 16 bytes, a row is row_bytes / 16 lanes.
template <bool ML>
__global__ __launch_bounds__(256) void gather_kernel(const GatherArgs a) {
  const int g = blockIdx.y;
  const int layer = ML ? (int)blockIdx.z / a.batch : 0;
  const int b = (int)blockIdx.z - layer * a.batch;
  const LayerView lv = layer_view<ML>(a, layer, 0);
  const int budget = a.gb.on ? a.gb.budget[g] : lv.budget;
  const gptr<const char> kb = lv.k;
  const gptr<const char> vb = lv.v;
  const int lanes_per_row = a.row_bytes >> 4;
  const int rows_per_pass = 256 / lanes_per_row;
  const int sub = threadIdx.x % lanes_per_row;
  const int r_in = threadIdx.x / lanes_per_row;
  const int s0 = a.cu[b];
  const int L = a.cu[b + 1] - s0;
  const int64_t obase = kept_base(a.gb, b, g, a.Hkv, budget);
  {
    const int r = blockIdx.x * rows_per_pass + r_in;
    if (r >= budget) return;
    const int j = lv.idx[obase + r];
    uint4 kv = make_uint4(0, 0, 0, 0), vv = make_uint4(0, 0, 0, 0);
    if (j >= 0 && j < L) {   // anything else is a dropped slot: zeros
      kv = load16(kb + (int64_t)(s0 + j) * a.k_stride_tok + (int64_t)g * a.k_stride_head +
                  16 * sub);
      vv = load16(vb + (int64_t)(s0 + j) * a.v_stride_tok + (int64_t)g * a.v_stride_head +
                  16 * sub);
    }
    const int64_t o = (obase + r) * a.row_bytes + 16 * sub;
    store16(lv.k_out + o, kv);
    store16(lv.v_out + o, vv);
  }
}

// Layer table entries from the host's compact form: pointers and budget as
// given, the SRH bit mask expanded into per-group head lists.  Grid (count),
// 256 threads.
__global__ __launch_bounds__(256) void put_layers_kernel(const PutArgs a) {
  const PutEntry &e = a.e[blockIdx.x];
  LayerDesc &d = a.table[a.first + blockIdx.x];
  const int tid = threadIdx.x;
  if (tid == 0) {
    d.q = e.q;
    d.k = e.k;
    d.v = e.v;
    d.scores = e.scores;
    d.idx = e.idx;
    d.k_out = e.k_out;
    d.v_out = e.v_out;
    d.budget = e.budget;
    d.reserved = 0;
  }
  // number of SRHs among query heads 0 .. x-1
  auto below = [&](int x) {
    int n = 0;
    for (int w = 0; w < (x >> 5); ++w) n += __popc(e.srh_bits[w]);
    if (x & 31) n += __popc(e.srh_bits[x >> 5] & ((1u << (x & 31)) - 1u));
    return n;
  };
  for (int h = tid; h < a.Hq; h += 256)
    if ((e.srh_bits[h >> 5] >> (h & 31)) & 1u) d.srh_head[below(h)] = (uint8_t)h;
  const int G = a.Hq / a.Hkv;
  for (int g = tid; g <= a.Hkv; g += 256) d.srh_off[g] = (uint16_t)below(g * G);
}

hipError_t launch_put_layers(const PutArgs &a, hipStream_t stream) {
  hipLaunchKernelGGL(put_layers_kernel, dim3(a.count), dim3(256), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_select(const SelectArgs &a, int n_layers, hipStream_t stream) {
  const int lb = a.batch * (n_layers > 0 ? n_layers : 1);
  if (a.sel_meta) {
    const dim3 slices(a.n_slices, a.n_sel, lb), sels(a.n_sel, lb);
    if (n_layers > 0) {
      hipLaunchKernelGGL(select_scan_kernel<true>, slices, dim3(kSelThreads), 0, stream, a);
      hipLaunchKernelGGL(select_resolve_kernel<true>, sels, dim3(kSelThreads), 0, stream, a);
      hipLaunchKernelGGL(select_write_kernel<true>, slices, dim3(kSelThreads), 0, stream, a);
    } else {
      hipLaunchKernelGGL(select_scan_kernel<false>, slices, dim3(kSelThreads), 0, stream, a);
      hipLaunchKernelGGL(select_resolve_kernel<false>, sels, dim3(kSelThreads), 0, stream, a);
      hipLaunchKernelGGL(select_write_kernel<false>, slices, dim3(kSelThreads), 0, stream, a);
    }
    return hipGetLastError();
  }
  if (n_layers > 0)
    hipLaunchKernelGGL(select_kernel<true>, dim3(a.n_sel, lb), dim3(kSelThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(select_kernel<false>, dim3(a.n_sel, lb), dim3(kSelThreads), 0, stream, a);
  return hipGetLastError();
}

// Layer-shared index set (section 3.3): the layer score of a prefix position
// is the mean over all the layer's SRHs of their pooled window sums, i.e. the
// per-group scores weighted by each group's SRH count; it replaces every
// group's row (window positions stay +inf).  Grid (ceil(max L / 256), batch
// [x layers]), 256 threads, one position per thread.
template <bool ML>
__global__ __launch_bounds__(256) void combine_kernel(const CombineArgs a) {
  const int layer = ML ? (int)blockIdx.y / a.batch : 0;
  const int b = (int)blockIdx.y - layer * a.batch;
  const LayerView lv = layer_view<ML>(a, layer, 0);
  const int s0 = a.cu[b];
  const int L = a.cu[b + 1] - s0;
  const int t = (int)blockIdx.x * 256 + (int)threadIdx.x;
  if (t >= L) return;
  const gptr<float> sc = lv.scores + s0 + t;
  float v = INFINITY;
  if (t < L - a.W) {
    float acc = 0.f;
    int n_total = 0;
    for (int g = 0; g < a.Hkv; ++g) {
      const int n = srh_count<ML>(a, layer, g);
      if (n) acc += (float)n * sc[(int64_t)g * a.T];
      n_total += n;
    }
    v = acc / (float)n_total;
  }
  for (int g = 0; g < a.Hkv; ++g) sc[(int64_t)g * a.T] = v;
}

hipError_t launch_combine(const CombineArgs &a, int n_layers, int lmax, hipStream_t stream) {
  const dim3 grid((lmax + 255) / 256, a.batch * (n_layers > 0 ? n_layers : 1));
  if (n_layers > 0)
    hipLaunchKernelGGL(combine_kernel<true>, grid, dim3(256), 0, stream, a);
  else
    hipLaunchKernelGGL(combine_kernel<false>, grid, dim3(256), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_gather(const GatherArgs &a, int n_layers, int max_budget, hipStream_t stream) {
  const int rows_per_block = 256 / (a.row_bytes >> 4);
  const int nblk = (max_budget + rows_per_block - 1) / rows_per_block;
  if (n_layers > 0)
    hipLaunchKernelGGL(gather_kernel<true>, dim3(nblk, a.Hkv, a.batch * n_layers), dim3(256), 0,
                       stream, a);
  else
    hipLaunchKernelGGL(gather_kernel<false>, dim3(nblk, a.Hkv, a.batch), dim3(256), 0, stream,
                       a);
  return hipGetLastError();
}

}  // namespace ckv
