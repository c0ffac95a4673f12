// Host launchers of the CompressKV kernels (defined next to the kernels).
#pragma once

#include "ckv_device.h"

namespace ckv {

// Enqueue the statistics and column-sum kernels; rt_max = max SRH row tiles of a group.
hipError_t launch_score(const ScoreArgs &a, int dtype_bf16, int head_dim, int rt_max, int batch,
                        hipStream_t stream);
// Multi-layer scoring: grid z = batch * n_layers, operands from a.layers.
hipError_t launch_score_layers(const ScoreArgs &a, int dtype_bf16, int head_dim, int rt_max,
                               int batch, int n_layers, hipStream_t stream);
// Selection and gather; n_layers > 0 reads the operands from the table
// (a.layers), n_layers == 0 from a.l0.
hipError_t launch_select(const SelectArgs &a, int n_layers, hipStream_t stream);
// Layer-shared index set: layer score into every group's row of the scores.
hipError_t launch_combine(const CombineArgs &a, int n_layers, int lmax, hipStream_t stream);
// Writes table entries [first, first + count) from a.e (count <= kPutLayers).
hipError_t launch_put_layers(const PutArgs &a, hipStream_t stream);

// Single-pass scoring (onepass_score.hip): bf16 keys, operands in the layer
// table.  Zeroes fill_ints ints from f.fill_base, then runs the main kernel on
// `grid` persistent workgroups, the catch-up kernel and the boundary kernel.
hipError_t launch_onepass(const OnePassArgs &f, int head_dim, int rt_max, int grid,
                          int64_t fill_ints, hipStream_t stream);
// max_budget: the largest budget over the layers (sizes the grid).
hipError_t launch_gather(const GatherArgs &a, int n_layers, int max_budget, hipStream_t stream);

}  // namespace ckv
