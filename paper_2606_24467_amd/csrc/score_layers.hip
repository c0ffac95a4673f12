// Scoring kernels (S1-S4) for the multi-layer entry point: grid z runs over
// (layer, sequence) pairs and the operands come from the layer table.
#include "ckv_launch.h"
#include "score_kernels.h"

namespace ckv {

hipError_t launch_score_layers(const ScoreArgs &a, int dtype_bf16, int head_dim, int rt_max,
                               int batch, int n_layers, hipStream_t stream) {
  return launch_score_any<true>(a, dtype_bf16, head_dim, rt_max, batch * n_layers, stream);
}

}  // namespace ckv
