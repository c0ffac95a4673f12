// Selection (S5) and eviction gather (S6) kernels of the CompressKV path.
//
// S5 keeps, per (sequence, KV group), the (budget - W) highest prefix scores
// (section 3.3: the N best tokens keep their KV pairs) with ties going to the
// lowest position, plus the W window positions, written in ascending order.
// Scores are non-negative floats, so their bit patterns order like unsigned
// integers: a three-digit radix select (11 + 11 + 10 bits) over LDS
// histograms finds the exact bit pattern of the k-th largest score, and an
// ordered compaction writes the kept positions.  Integer work only, so the
// result does not depend on scheduling.
//
// S6 copies the kept K and V rows (section 3.3: the retained KV pairs form the
// compressed cache) with 16-byte lanes; rows whose index is -1 become zeros.
#include "ckv_device.h"

namespace ckv {

constexpr int kSelThreads = 1024;

// Inclusive prefix sum over the 1024 threads of the block.
__device__ __forceinline__ int block_inclusive_scan(int x, int *lds_waves) {
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
  __syncthreads();   // lds_waves is reused by the next scan
  return x + before;
}

// Grid (Hkv, batch), 1024 threads.
__global__ __launch_bounds__(kSelThreads) void select_kernel(const SelectArgs a) {
  const int g = blockIdx.x, b = blockIdx.y;
  const int tid = threadIdx.x;
  const int s0 = a.cu[b];
  const int L = a.cu[b + 1] - s0;
  int32_t *out = a.idx + ((int64_t)b * a.Hkv + g) * a.budget;
  if (L <= a.budget) {
    for (int j = tid; j < a.budget; j += kSelThreads) out[j] = (j < L) ? j : -1;
    return;
  }
  const int P = L - a.W;
  const int k = a.budget - a.W;     // prefix tokens to keep, 0 <= k < P
  for (int w = tid; w < a.W; w += kSelThreads) out[k + w] = P + w;
  if (k == 0) return;
  const uint32_t *sc = reinterpret_cast<const uint32_t *>(a.scores + (int64_t)g * a.T + s0);

  __shared__ int hist[2048];
  __shared__ int scan_tmp[kSelThreads / 64];
  __shared__ int bucket_s, remain_s;
  uint32_t prefix = 0, pmask = 0;
  int remain = k;                   // rank of the target inside the current prefix
  const int shifts[3] = {21, 10, 0};
  const int widths[3] = {11, 11, 10};
  for (int pass = 0; pass < 3; ++pass) {
    const int sh = shifts[pass];
    const uint32_t dmask = (1u << widths[pass]) - 1u;
    const int nb = 1 << widths[pass];
    for (int i = tid; i < 2048; i += kSelThreads) hist[i] = 0;
    __syncthreads();
    for (int j = tid; j < P; j += kSelThreads) {
      const uint32_t u = sc[j];
      if ((u & pmask) == prefix) atomicAdd(&hist[(u >> sh) & dmask], 1);
    }
    __syncthreads();
    // Counts from the top bucket down: thread t owns buckets nb-1-2t and nb-2-2t.
    const int hi_b = nb - 1 - 2 * tid;
    int c_hi = 0, c_lo = 0;
    if (hi_b >= 0) c_hi = hist[hi_b];
    if (hi_b - 1 >= 0) c_lo = hist[hi_b - 1];
    const int incl = block_inclusive_scan(c_hi + c_lo, scan_tmp);
    const int excl = incl - c_hi - c_lo;   // elements in buckets above hi_b
    if (hi_b >= 0) {
      if (excl < remain && remain <= excl + c_hi) {
        bucket_s = hi_b;
        remain_s = remain - excl;
      } else if (hi_b - 1 >= 0 && excl + c_hi < remain && remain <= excl + c_hi + c_lo) {
        bucket_s = hi_b - 1;
        remain_s = remain - excl - c_hi;
      }
    }
    __syncthreads();
    prefix |= (uint32_t)bucket_s << sh;
    pmask |= dmask << sh;
    remain = remain_s;
    __syncthreads();
  }
  // prefix is the exact bit pattern of the k-th largest score; `remain` of the
  // positions holding it are kept (the lowest ones), plus every larger score.
  const uint32_t thr = prefix;
  const int ept = (P + kSelThreads - 1) / kSelThreads;
  const int j0 = min(P, tid * ept), j1 = min(P, j0 + ept);
  int n_gt = 0, n_eq = 0;
  for (int j = j0; j < j1; ++j) {
    const uint32_t u = sc[j];
    n_gt += (u > thr);
    n_eq += (u == thr);
  }
  const int eq_before = block_inclusive_scan(n_eq, scan_tmp) - n_eq;
  const int take_eq = max(0, min(n_eq, remain - eq_before));
  const int n_sel = n_gt + take_eq;
  int pos = block_inclusive_scan(n_sel, scan_tmp) - n_sel;
  int eq_left = take_eq;
  for (int j = j0; j < j1; ++j) {
    const uint32_t u = sc[j];
    bool keep = (u > thr);
    if (u == thr && eq_left > 0) {
      keep = true;
      --eq_left;
    }
    if (keep && pos < k) out[pos++] = j;   // bound holds for finite scores; guards NaN input
  }
}

// Grid (ceil(budget / rows_per_block), Hkv, batch), 256 threads; each lane
// moves 16 bytes, a row is row_bytes / 16 lanes.
__global__ __launch_bounds__(256) void gather_kernel(const GatherArgs a) {
  const int g = blockIdx.y, b = blockIdx.z;
  const int lanes_per_row = a.row_bytes >> 4;
  const int rows_per_pass = 256 / lanes_per_row;
  const int sub = threadIdx.x % lanes_per_row;
  const int r_in = threadIdx.x / lanes_per_row;
  const int s0 = a.cu[b];
  const int L = a.cu[b + 1] - s0;
  const int64_t obase = ((int64_t)b * a.Hkv + g) * a.budget;
  const int r_first = blockIdx.x * 4 * rows_per_pass;
  for (int p = 0; p < 4; ++p) {
    const int r = r_first + p * rows_per_pass + r_in;
    if (r >= a.budget) break;
    const int j = a.idx[obase + r];
    uint4 kv = make_uint4(0, 0, 0, 0), vv = make_uint4(0, 0, 0, 0);
    if (j >= 0 && j < L) {   // anything else is a dropped slot: zeros
      kv = load16(a.k + (int64_t)(s0 + j) * a.k_stride_tok + (int64_t)g * a.k_stride_head +
                  16 * sub);
      vv = load16(a.v + (int64_t)(s0 + j) * a.v_stride_tok + (int64_t)g * a.v_stride_head +
                  16 * sub);
    }
    const int64_t o = (obase + r) * a.row_bytes + 16 * sub;
    *reinterpret_cast<uint4 *>(a.k_out + o) = kv;
    *reinterpret_cast<uint4 *>(a.v_out + o) = vv;
  }
}

hipError_t launch_select(const SelectArgs &a, int batch, hipStream_t stream) {
  hipLaunchKernelGGL(select_kernel, dim3(a.Hkv, batch), dim3(kSelThreads), 0, stream, a);
  return hipGetLastError();
}

hipError_t launch_gather(const GatherArgs &a, int batch, hipStream_t stream) {
  const int rows_per_block = 4 * (256 / (a.row_bytes >> 4));
  const int nblk = (a.budget + rows_per_block - 1) / rows_per_block;
  hipLaunchKernelGGL(gather_kernel, dim3(nblk, a.Hkv, batch), dim3(256), 0, stream, a);
  return hipGetLastError();
}

}  // namespace ckv
