// Host-side dispatch of a step's launches to the kernel translation units by
// block size and error-feedback format.
#include "step_kernel.h"

namespace microadam {

size_t step_lds_bytes(int block, int k_full, int value_f32) {
  (void)k_full;
  (void)value_f32;
  if (block > kSubBlock) return update_large_lds();
  const size_t sel = select_lds_words() * 4;
  const size_t upd = update_lds_max(threads_for_block(block));
  return sel > upd ? sel : upd;
}

hipError_t launch_select(const StepParams& p, int grad_bf16, int value_f32, int64_t first, int64_t count,
                         hipStream_t stream) {
  if (count <= 0) return hipSuccess;
  if (p.block > kSubBlock) {
    switch (p.ef_mode) {
      case 0: return launch_select_large_near4(p, grad_bf16, value_f32, first, count, stream);
      case 1: return launch_select_large_near8(p, grad_bf16, value_f32, first, count, stream);
      case 2: return launch_select_large_rand4(p, grad_bf16, value_f32, first, count, stream);
      case 3: return launch_select_large_rand8(p, grad_bf16, value_f32, first, count, stream);
      default: return hipErrorInvalidValue;
    }
  }
  switch (p.ef_mode) {
    case 0: return launch_select_near4(p, grad_bf16, value_f32, first, count, stream);
    case 1: return launch_select_near8(p, grad_bf16, value_f32, first, count, stream);
    case 2: return launch_select_rand4(p, grad_bf16, value_f32, first, count, stream);
    case 3: return launch_select_rand8(p, grad_bf16, value_f32, first, count, stream);
    default: return hipErrorInvalidValue;
  }
}

size_t fused_lds_bytes(int value_f32) {
  return (value_f32 ? step_kernel_lds_words<true>() : step_kernel_lds_words<false>()) * 4;
}

hipError_t launch_step(const StepParams& p, int bf16, int value_f32, int64_t first, int64_t count,
                       hipStream_t stream) {
  if (count <= 0) return hipSuccess;
  switch (p.ef_mode) {
    case 0: return launch_step_near4(p, bf16, value_f32, first, count, stream);
    case 1: return launch_step_near8(p, bf16, value_f32, first, count, stream);
    case 2: return launch_step_rand4(p, bf16, value_f32, first, count, stream);
    case 3: return launch_step_rand8(p, bf16, value_f32, first, count, stream);
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_update(const StepParams& p, int param_bf16, int value_f32, int64_t first, int64_t count,
                         hipStream_t stream) {
  if (count <= 0) return hipSuccess;
  if (p.block > kSubBlock) return launch_update_large_blocks(p, param_bf16, value_f32, first, count, stream);
  return launch_update_blocks(p, param_bf16, value_f32, first, count, stream);
}

hipError_t launch_moments(const StepParams& p, int64_t first_block, int64_t num_blocks, float* mhat,
                          float* vhat, int value_f32, hipStream_t stream) {
  if (num_blocks <= 0) return hipSuccess;
  if (p.block > kSubBlock)
    return launch_moments_large_blocks(p, first_block, num_blocks, mhat, vhat, value_f32, stream);
  return launch_moments_blocks(p, first_block, num_blocks, mhat, vhat, value_f32, stream);
}

}  // namespace microadam
