// The multi-wave select kernel for blocks above 4096 elements, 4-bit codes, round to nearest.
#include "select_large_kernel.h"

namespace microadam {

hipError_t launch_select_large_near4(const StepParams& p, int grad_bf16, int value_f32, int64_t first, int64_t count,
                                  hipStream_t stream) {
  return launch_select_large_mode<0>(p, grad_bf16, value_f32, first, count, stream);
}

}  // namespace microadam
