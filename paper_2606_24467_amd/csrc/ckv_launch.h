// Host launchers of the CompressKV kernels (defined next to the kernels).
#pragma once

#include "ckv_device.h"

namespace ckv {

// Enqueue the statistics and column-sum kernels; rt_max = max SRH row tiles of a group.
hipError_t launch_score(const ScoreArgs &a, int dtype_bf16, int head_dim, int rt_max, int batch,
                        hipStream_t stream);
hipError_t launch_select(const SelectArgs &a, int batch, hipStream_t stream);

// Single-pass scoring (fused_score.hip).
struct FusedArgs;
constexpr int kFusedMaxBatch = 64;
hipError_t launch_fused_score(const FusedArgs &f, int dtype_bf16, int head_dim, int rt_max,
                              int unit_tiles, int counters, hipStream_t stream);
int fused_resident_workgroups(int dtype_bf16, int head_dim, int rt_max, int unit_tiles);
hipError_t launch_gather(const GatherArgs &a, int batch, hipStream_t stream);

}  // namespace ckv
