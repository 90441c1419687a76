// The multi-wave select kernel for blocks above 4096 elements, 8-bit codes, randomized rounding (Lemma 1).
#include "select_large_kernel.h"

namespace microadam {

hipError_t launch_select_large_rand8(const StepParams& p, int grad_bf16, int value_f32, int64_t first, int64_t count,
                                  hipStream_t stream) {
  return launch_select_large_mode<kEf8 | kEfRandom>(p, grad_bf16, value_f32, first, count, stream);
}

}  // namespace microadam
