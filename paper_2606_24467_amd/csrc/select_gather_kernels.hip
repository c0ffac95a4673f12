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
constexpr int kCandCap = 4096;               // candidates of the first-digit bucket kept in LDS
constexpr int kEpt = 32;                     // scores per thread held in registers per round
constexpr int kRound = kSelThreads * kEpt;   // scores per round

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
// owns a run of kWaveRun consecutive positions and its lanes take
// consecutive positions for each e, so a load instruction reads 256
// contiguous bytes and the position order is (wave, e, lane).
constexpr int kWaveRun = 64 * kEpt;
__device__ __forceinline__ int elem_pos(int r0, int e) {
  return r0 + (int)(threadIdx.x >> 6) * kWaveRun + e * 64 + (int)(threadIdx.x & 63);
}

// Lanes below this one whose bit is set in m.
__device__ __forceinline__ int lanes_below(unsigned long long m) {
  return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                        __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

// A thread's kEpt scores of the round starting at r0 into registers (all
// loads issued together); positions >= P read as 0 and are masked by the
// callers.
__device__ __forceinline__ void load_round(gptr<const uint32_t> sc, int P, int r0,
                                           uint32_t (&v)[kEpt]) {
#pragma unroll
  for (int e = 0; e < kEpt; ++e) {
    const int j = elem_pos(r0, e);
    v[e] = (j < P) ? sc[j] : 0u;
  }
}

// Grid (Hkv, batch [x layers]), 1024 threads.
template <bool ML>
__global__ __launch_bounds__(kSelThreads) void select_kernel(const SelectArgs a) {
  const int g = blockIdx.x;         // selection index: the KV group, or 0 (layer-shared set)
  const int layer = ML ? (int)blockIdx.y / a.batch : 0;
  const int b = (int)blockIdx.y - layer * a.batch;
  const LayerView lv = layer_view<ML>(a, layer, 0);
  const int budget = a.gb.on ? a.gb.budget[g] : lv.budget;
  const int tid = threadIdx.x;
  const int s0 = a.cu[b];
  const int L = a.cu[b + 1] - s0;
  const gptr<int32_t> out = lv.idx + kept_base(a.gb, b, g, a.Hkv, budget);
  // position `pos` of the kept list, in every idx row this selection serves
  auto put = [&](int pos, int32_t val) {
    for (int r = 0; r < a.out_groups; ++r) out[(int64_t)r * budget + pos] = val;
  };
  if (L <= budget) {
    for (int j = tid; j < budget; j += kSelThreads) put(j, (j < L) ? j : -1);
    return;
  }
  const int P = L - a.W;
  const int k = budget - a.W;       // prefix tokens to keep, 0 <= k < P
  for (int w = tid; w < a.W; w += kSelThreads) put(k + w, P + w);
  if (k == 0) return;
  const gptr<const uint32_t> sc =
      reinterpret_cast<gptr<const uint32_t>>(lv.scores + (int64_t)g * a.T + s0);
  const int nrounds = (P + kRound - 1) / kRound;
  const bool resident = (nrounds == 1);   // scores stay in registers for every pass

  __shared__ int hist[kHistBins];
  __shared__ int scan_tmp[kSelThreads / 64];
  __shared__ int wave_cnt[2][kSelThreads / 64];
  __shared__ int bucket_s, remain_s, ncand_s;
  __shared__ uint32_t cand_u[kCandCap];
  __shared__ int cand_j[kCandCap];

  uint32_t v[kEpt];
  if (resident) load_round(sc, P, 0, v);

  // Digit 1: bits 30..20.
  if (a.hist) {
    const int *hg = a.hist + layer * a.hist_layer + ((int64_t)b * a.Hkv + g) * kHistBins;
    for (int i = tid; i < kHistBins; i += kSelThreads) hist[i] = hg[i];
  } else {
    for (int i = tid; i < kHistBins; i += kSelThreads) hist[i] = 0;
    __syncthreads();
    for (int r = 0; r < nrounds; ++r) {
      if (!resident) load_round(sc, P, r * kRound, v);
#pragma unroll
      for (int e = 0; e < kEpt; ++e) hist_add(hist, hist_bin(v[e]), elem_pos(r * kRound, e) < P);
    }
  }
  if (tid == 0) ncand_s = 0;
  __syncthreads();
  find_bucket(hist, kHistBins, k, scan_tmp, &bucket_s, &remain_s);
  uint32_t pmask = 0x7FFu << 20;
  uint32_t prefix = (uint32_t)bucket_s << 20;
  int remain = remain_s;

  // Candidates: prefix elements whose first digit equals the chosen bucket.
  for (int r = 0; r < nrounds; ++r) {
    if (!resident) load_round(sc, P, r * kRound, v);
#pragma unroll
    for (int e = 0; e < kEpt; ++e) {
      const int j = elem_pos(r * kRound, e);
      if (j < P && (v[e] & pmask) == prefix) {
        const int slot = atomicAdd(&ncand_s, 1);
        if (slot < kCandCap) {
          cand_u[slot] = v[e];
          cand_j[slot] = j;
        }
      }
    }
  }
  __syncthreads();
  const int nc = ncand_s;
  const bool in_lds = nc <= kCandCap;

  // Digits 2 (bits 19..9) and 3 (bits 8..0) on the candidates (or, if they
  // overflow the LDS list, on every prefix element that matches so far).
  const int shifts[2] = {9, 0};
  const int widths[2] = {11, 9};
  for (int pass = 0; pass < 2; ++pass) {
    const int sh = shifts[pass];
    const uint32_t dmask = (1u << widths[pass]) - 1u;
    for (int i = tid; i < kHistBins; i += kSelThreads) hist[i] = 0;
    __syncthreads();
    if (in_lds) {
      for (int base = 0; base < nc; base += kSelThreads) {
        const int i = base + tid;
        const uint32_t u = (i < nc) ? cand_u[i] : 0u;
        hist_add(hist, (int)((u >> sh) & dmask), i < nc && (u & pmask) == prefix);
      }
    } else {
      for (int r = 0; r < nrounds; ++r) {
        if (!resident) load_round(sc, P, r * kRound, v);
#pragma unroll
        for (int e = 0; e < kEpt; ++e)
          hist_add(hist, (int)((v[e] >> sh) & dmask),
                   elem_pos(r * kRound, e) < P && (v[e] & pmask) == prefix);
      }
    }
    __syncthreads();
    find_bucket(hist, 1 << widths[pass], remain, scan_tmp, &bucket_s, &remain_s);
    prefix |= (uint32_t)bucket_s << sh;
    pmask |= dmask << sh;
    remain = remain_s;
    __syncthreads();
  }

  // prefix is the exact bit pattern of the k-th largest score; `remain` of the
  // positions holding it are kept (the lowest ones), plus every larger score.
  // Ordered compaction, round by round: each wave counts its elements above
  // and at the threshold, every wave forms the prefix over the waves before
  // it, and the kept positions are written in (wave, e, lane) order.
  const uint32_t thr = prefix;
  const int lane = tid & 63, wave = tid >> 6;
  int pos_base = 0, eq_base = 0;
  for (int r = 0; r < nrounds; ++r) {
    if (!resident) load_round(sc, P, r * kRound, v);
    int n_gt = 0, n_eq = 0;   // this thread's counts, then the wave's
#pragma unroll
    for (int e = 0; e < kEpt; ++e) {
      const uint32_t u = v[e] & 0x7FFFFFFFu;
      const bool ok = elem_pos(r * kRound, e) < P;
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
    for (int e = 0; e < kEpt; ++e) {
      const int j = elem_pos(r * kRound, e);
      const uint32_t u = v[e] & 0x7FFFFFFFu;
      const bool ok = j < P;
      const bool gt = ok && u > thr, eq = ok && u == thr;
      const unsigned long long m_gt = __ballot(gt), m_eq = __ballot(eq);
      if ((m_gt | m_eq) == 0ull) continue;   // nothing kept at this e (uniform; most e)
      const bool keep = gt || (eq && eq_rank + lanes_below(m_eq) < remain);
      const unsigned long long m_keep = __ballot(keep);
      const int my_pos = pos + lanes_below(m_keep);
      if (keep && my_pos < k) put(my_pos, j);   // bound holds for finite scores; guards NaN
      pos += __popcll(m_keep);
      eq_rank += __popcll(m_eq);
    }
    eq_base += eq_total;
    pos_base += sel_total;
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
  if (n_layers > 0)
    hipLaunchKernelGGL(select_kernel<true>, dim3(a.n_sel, a.batch * n_layers), dim3(kSelThreads),
                       0, stream, a);
  else
    hipLaunchKernelGGL(select_kernel<false>, dim3(a.n_sel, a.batch), dim3(kSelThreads), 0, stream,
                       a);
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
