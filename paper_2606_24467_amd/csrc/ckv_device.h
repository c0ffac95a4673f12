// Device-side building blocks of the CompressKV eviction kernels (gfx950).
//
// Operand layout used by every scoring kernel.  One wavefront (64 lanes)
// multiplies a 16-row tile of one matrix with a 16-row tile of another along
// the head dimension D with v_mfma_f32_16x16x32_bf16 (bf16) or
// v_mfma_f32_16x16x4_f32 (fp32).  Lane l = 16*quad + c holds row c of each
// operand tile; for the 16-byte slice s of a row it holds bytes
// [64*s + 16*quad, 64*s + 16*quad + 16).  A and B use the same slicing, so the
// pairing of reduction indices is consistent and the MFMA returns plain dot
// products.  The 16x16 result is held as: lane l, element r = C[4*quad + r][c],
// where the first index runs over the A rows and the second over the B rows.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace ckv {

constexpr int kMaxKvHeads = 128;
constexpr int kMaxQHeads = 256;
constexpr int kMaxPoolKernel = 31;   // pooling halo (k-1)/2 <= 15 fits one 16-key tile
constexpr int kMaxChunk2 = 1024;     // keys per column-sum workgroup (LDS column sums)
constexpr int kHistBins = 2048;      // first radix digit of the selection: value bits 30..20

// Scores are non-negative floats, ordered like their bit patterns; the first
// selection digit is the exponent and the top three mantissa bits.
__device__ __forceinline__ int hist_bin(uint32_t u) { return (int)((u >> 20) & 0x7FFu); }

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

// Operands of one layer.  Single-layer calls pass one inline in the kernel
// arguments; the multi-layer entry point keeps a table of them in device
// memory (written by put_layers_kernel) and the kernels index it by layer.
struct alignas(16) LayerDesc {
  const void *q;          // [batch, W, Hq, D]
  const void *k, *v;      // [T, Hkv, D] with the problem's strides (elements)
  float *scores;          // [Hkv][T]
  int32_t *idx;           // [batch][Hkv][budget]
  void *k_out, *v_out;    // [batch][Hkv][budget][D]
  int32_t budget;
  int32_t reserved;
  uint16_t srh_off[kMaxKvHeads + 2];   // SRHs of group g: srh_head[srh_off[g] .. srh_off[g+1])
  uint8_t srh_head[kMaxQHeads];        // query-head indices, ascending within a group
};
static_assert(offsetof(LayerDesc, srh_off) % 4 == 0 && offsetof(LayerDesc, srh_head) % 4 == 0,
              "table fields read as 32-bit words");

// Pointers into global memory.  Pointers read from the layer table have no
// address space the compiler can infer; generic (flat) accesses would share
// the wait counter of the LDS reads and serialise every key load with them.
template <typename T>
using gptr = __attribute__((address_space(1))) T *;
template <typename T>
__device__ __forceinline__ gptr<T> to_global(T *p) {
  return (gptr<T>)p;
}

// Read-only during a kernel (the layer table, the sequence offsets): uniform
// loads through the constant address space become scalar loads.
template <typename T>
using cptr = const __attribute__((address_space(4))) T *;
template <typename T>
__device__ __forceinline__ cptr<T> to_const(const T *p) {
  return (cptr<T>)p;
}

// srh_off[g] of a table entry through aligned 32-bit reads of the constant
// address space (16-bit fields can not be read by scalar loads); for a
// uniform (layer, g) these stay scalar and never wait on a kernel's vector
// loads.
__device__ __forceinline__ int srh_off_at(cptr<LayerDesc> d, int g) {
  const cptr<uint32_t> w =
      reinterpret_cast<cptr<uint32_t>>(reinterpret_cast<cptr<char>>(d) + offsetof(LayerDesc, srh_off));
  return (int)((w[g >> 1] >> (16 * (g & 1))) & 0xFFFFu);
}

// What a workgroup uses of its layer, as global pointers; off / nsrh describe
// the SRHs of group g (srh_head[off .. off + nsrh)).
struct LayerView {
  gptr<const char> q, k, v;
  gptr<float> scores;
  gptr<int32_t> idx;
  gptr<char> k_out, v_out;
  gptr<const uint8_t> srh_head;
  int budget, off, nsrh;
};

// The layer a workgroup works on: the inline one, or entry `layer` of the table.
template <bool ML, typename A>
__device__ __forceinline__ LayerView layer_view(const A &a, int layer, int g) {
  LayerView v;
  if constexpr (ML) {
    cptr<LayerDesc> d = to_const(a.layers) + layer;
    v.q = to_global(static_cast<const char *>(d->q));
    v.k = to_global(static_cast<const char *>(d->k));
    v.v = to_global(static_cast<const char *>(d->v));
    v.scores = to_global(d->scores);
    v.idx = to_global(d->idx);
    v.k_out = to_global(static_cast<char *>(d->k_out));
    v.v_out = to_global(static_cast<char *>(d->v_out));
    v.srh_head = &(to_global(a.layers) + layer)->srh_head[0];
    v.budget = d->budget;
    v.off = srh_off_at(d, g);
    v.nsrh = srh_off_at(d, g + 1) - v.off;
  } else {
    (void)layer;
    const LayerDesc &d = a.l0;
    v.q = to_global(static_cast<const char *>(d.q));
    v.k = to_global(static_cast<const char *>(d.k));
    v.v = to_global(static_cast<const char *>(d.v));
    v.scores = to_global(d.scores);
    v.idx = to_global(d.idx);
    v.k_out = to_global(static_cast<char *>(d.k_out));
    v.v_out = to_global(static_cast<char *>(d.v_out));
    v.srh_head = to_global(&d.srh_head[0]);
    v.budget = d.budget;
    v.off = d.srh_off[g];
    v.nsrh = d.srh_off[g + 1] - v.off;
  }
  return v;
}

// SRHs of group g of the layer.
template <bool ML, typename A>
__device__ __forceinline__ int srh_count(const A &a, int layer, int g) {
  if constexpr (ML) {
    cptr<LayerDesc> d = to_const(a.layers) + layer;
    return srh_off_at(d, g + 1) - srh_off_at(d, g);
  } else {
    (void)layer;
    return a.l0.srh_off[g + 1] - a.l0.srh_off[g];
  }
}

// Arguments of the scoring kernels.
struct ScoreArgs {
  LayerDesc l0;            // single-layer calls
  const LayerDesc *layers; // multi-layer calls: [n_layers]
  const int32_t *cu;       // [batch+1] sequence offsets
  float2 *stats;           // per layer: [batch][Hkv][parts_stride][row_slots] partial (ref, sum)
  int64_t stats_layer;     // float2 elements between layers
  int *hist;               // per layer: [batch][Hkv][kHistBins] first selection digit counts
  int64_t hist_layer;      // ints between layers
  int64_t k_stride_tok, k_stride_head;
  int32_t T, batch, Hq, Hkv, W;
  int32_t th;             // 16-row tiles per SRH: ceil(W / 16)
  int32_t row_slots;      // padded rows per (sequence, group, chunk) in stats
  int32_t chunk1, max_chunks1;   // keys per statistics chunk, chunks of the longest sequence
  int32_t parts_stride;          // partial slots per (sequence, group) in stats
  int32_t chunk2, max_chunks2;   // keys per column-sum chunk, chunks of the longest sequence
  int32_t cpw1, cpw2;            // consecutive chunks per leading workgroup (statistics, column sums)
  int32_t lead1, lead2;          // leading workgroups per (sequence, group) and layer; the
                                 // chunks after lead * cpw go one per workgroup
  int32_t nz;                    // sequences x layers of the launch (set by the launcher)
  float c1;               // softmax scale * log2(e): logits in base-2 units
  int32_t pool_kernel, pool_type, reduce_order;
  uint32_t head_end_mask;  // bit rt set if row tile rt is the last tile of an SRH
  // Both passes in one launch (score_kernels.h, fused_kernel); null: two launches.
  int *fused_skip;         // [0]: entries, then the workgroups left to the catch-up kernel
  int32_t fused_spin;      // polls of a group's normalisers before a workgroup leaves its
                           // column sums to the catch-up kernel (< 0: all of them)
  int *fused_arrive;       // [segments] statistics workgroups of a segment that have published
  float2 *fused_bias;      // [segments][row_slots] (normaliser, -1) once published
};

// Workgroups per (sequence, group) and pass of the fused two-pass launch, and
// its grid (8 XCDs x 2 passes x kFusedMembers per 8 (sequence, group) pairs;
// nz sequences x layers).
constexpr int kFusedMembers = 32;
__host__ __device__ inline int64_t fused_blocks(int Hkv, int nz) {
  return (int64_t)kFusedMembers * 8 * 2 * (((int64_t)Hkv * nz + 7) / 8);
}

// Arguments of the single-pass scoring kernels (operands in the layer table:
// the launch covers table layers 0 .. n_layers - 1).
constexpr int kOnePassUnitKeys = 256;   // keys of one unit
constexpr int kOnePassMaxBatch = 64;
struct OnePassArgs {
  ScoreArgs s;             // s.stats: unit partials [layer][group][unit][row] (max, -sum)
  int *fill_base;          // start of the block zeroed before the launch
  int *ticket;             // next unit to take
  int *skip_count;         // units left to the catch-up kernel
  int *arrive;             // [layers][batch * Hkv] units of each segment that have published
  float2 *bias;            // [layers][batch * Hkv][row_slots] (normaliser, 1) once published
  int *skip_list;          // [n_units_total]
  float *edges;            // [n_units_total][heads_max][2][ew] window sums at each unit's ends
  int n_units_total;       // units of all layers of the launch
  int units_per_layer;     // seq_units[batch]
  int seq_units[kOnePassMaxBatch + 1];   // first ticket of sequence b within a layer
  int spin_limit;          // polls of a late normaliser before the unit is left to catch-up
  int ew;                  // pool_kernel - 1: window sums kept at each end of a unit
  int heads_max;           // most SRHs in one group
};

// Per-group budgets (head-level allocation): group g keeps budget[g] rows,
// stored ragged: entry j of (sequence b, group g) is row b * total + off[g] + j.
struct GroupBudgets {
  int32_t on;
  int32_t total;                    // sum of the budgets
  int32_t budget[kMaxKvHeads];
  int32_t off[kMaxKvHeads];         // exclusive prefix sums
};

// Where (sequence b, group g)'s kept list starts in idx (rows of the
// compact cache), and its budget.
__device__ __forceinline__ int64_t kept_base(const GroupBudgets &gb, int b, int g, int Hkv,
                                             int budget) {
  return gb.on ? (int64_t)b * gb.total + gb.off[g] : ((int64_t)b * Hkv + g) * budget;
}

struct SelectArgs {
  LayerDesc l0;            // uses scores, idx, budget
  const LayerDesc *layers;
  const int *hist;         // per layer [batch][Hkv][kHistBins], or NULL (then counted here)
  int64_t hist_layer;
  const int32_t *cu;
  int32_t T, Hkv, W, batch;
  int32_t n_sel;           // selections per (layer, sequence): Hkv, or 1 (layer-shared set)
  int32_t out_groups;      // idx rows each selection writes: 1, or Hkv (layer-shared set)
  GroupBudgets gb;         // per-group budgets (single-layer calls), if gb.on
  // Split selection (sequences longer than one slice; needs hist): per
  // selection kSelMetaPerSlice * n_slices meta words, n_slices lists of
  // cand_cap candidate scores and n_slices lists of cand_cap (position,
  // score) pairs; NULL sel_meta selects one workgroup per selection.
  int *sel_meta;
  uint32_t *sel_cand;
  uint64_t *sel_ord;   // (score bits << 32) | position, bit 31 marking a candidate
  int32_t n_slices, cand_cap;
};

constexpr int kSelSlice = 32768;       // positions per slice of the split selection
constexpr int kMaxSelSlices = 64;      // longest prefix it takes: 64 slices
constexpr int kSelSliceCap = kSelSlice;   // list entries kept per slice: all its positions
// Meta words per slice of a split selection: candidates, the 16 waves' list
// lengths, the slice's first kept-list position, ties in the slices before,
// the threshold and the ties kept.
constexpr int kSelMetaPerSlice = 21;

// Layer-shared index set: the layer score from the per-group scores.
struct CombineArgs {
  LayerDesc l0;            // uses scores, srh_off
  const LayerDesc *layers;
  const int32_t *cu;
  int32_t T, Hkv, W, batch;
};

struct GatherArgs {
  LayerDesc l0;            // uses k, v, idx, k_out, v_out, budget
  const LayerDesc *layers;
  const int32_t *cu;
  int64_t k_stride_tok, k_stride_head, v_stride_tok, v_stride_head;  // bytes
  int32_t Hkv, batch, row_bytes;
  GroupBudgets gb;         // per-group budgets (single-layer calls), if gb.on
};

// One layer of the table as the host hands it over (SRH mask as bits over the
// query heads); put_layers_kernel expands the mask into per-group lists.
constexpr int kPutLayers = 32;   // ~3.1 KB of kernel arguments: one launch for up to 32 layers
struct PutEntry {
  const void *q, *k, *v;
  float *scores;
  int32_t *idx;
  void *k_out, *v_out;
  int32_t budget;
  uint32_t srh_bits[kMaxQHeads / 32];
};
struct PutArgs {
  LayerDesc *table;
  int32_t first, count, Hq, Hkv;
  PutEntry e[kPutLayers];
};

// 16-byte slices per row per quad: D * sizeof(T) / 64.
template <typename T, int D>
struct Slices {
  static constexpr int n = D * (int)sizeof(T) / 64;
};

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint4 load16(gptr<const char> p) {
  return __builtin_bit_cast(uint4, *reinterpret_cast<gptr<const u32x4>>(p));
}

__device__ __forceinline__ void store16(gptr<char> p, uint4 v) {
  *reinterpret_cast<gptr<u32x4>>(p) = __builtin_bit_cast(u32x4, v);
}

// acc += A_tile * B_tile^T over one 16-byte slice of each row.
template <typename T>
__device__ __forceinline__ f32x4 mfma_slice(uint4 a, uint4 b, f32x4 acc);

template <>
__device__ __forceinline__ f32x4 mfma_slice<__bf16>(uint4 a, uint4 b, f32x4 acc) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), acc, 0, 0, 0);
}

template <>
__device__ __forceinline__ f32x4 mfma_slice<float>(uint4 a, uint4 b, f32x4 acc) {
  float4 fa = __builtin_bit_cast(float4, a);
  float4 fb = __builtin_bit_cast(float4, b);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(fa.x, fb.x, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(fa.y, fb.y, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(fa.z, fb.z, acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(fa.w, fb.w, acc, 0, 0, 0);
  return acc;
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }
__device__ __forceinline__ float fast_log2(float x) { return __builtin_amdgcn_logf(x); }

// Merge two (reference, sum) pairs, sum_i exp2(y_i - ref), into one.
__device__ __forceinline__ void merge_stats(float &ref, float &sum, float ref_o, float sum_o) {
  float m = fmaxf(ref, ref_o);
  if (m == -INFINITY) {
    sum = 0.f;
  } else {
    sum = sum * fast_exp2(ref - m) + sum_o * fast_exp2(ref_o - m);
  }
  ref = m;
}

}  // namespace ckv
