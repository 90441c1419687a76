// The fused step kernel for blocks of 2049 to 4096 elements, 4-bit codes, round to nearest (the paper's format).
#include "step_kernel.h"

namespace microadam {

hipError_t launch_step_near4(const StepParams& p, int bf16, int value_f32, int64_t first, int64_t count,
                             hipStream_t stream) {
  return launch_step_mode<0>(p, bf16, value_f32, first, count, stream);
}

}  // namespace microadam
