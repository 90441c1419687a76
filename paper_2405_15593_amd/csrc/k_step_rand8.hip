// The fused step kernel for blocks of 2049 to 4096 elements, 8-bit codes, randomized rounding (Lemma 1).
#include "step_kernel.h"

namespace microadam {

hipError_t launch_step_rand8(const StepParams& p, int bf16, int value_f32, int64_t first, int64_t count,
                             hipStream_t stream) {
  return launch_step_mode<kEf8 | kEfRandom>(p, bf16, value_f32, first, count, stream);
}

}  // namespace microadam
