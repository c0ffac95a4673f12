// Scoring kernels (S1-S4) for single-layer calls: operands in the arguments.
#include "ckv_launch.h"
#include "score_kernels.h"

namespace ckv {

hipError_t launch_score(const ScoreArgs &a, int dtype_bf16, int head_dim, int rt_max, int batch,
                        hipStream_t stream) {
  return launch_score_any<false>(a, dtype_bf16, head_dim, rt_max, batch, stream);
}

}  // namespace ckv
