// Types shared by the host side of libmicroadam and its HIP kernels.
// Internal to the library: the public interface is include/microadam.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace microadam {

constexpr int kMaxWindow = 64;       // largest supported window m
constexpr int kMaxBlock = 65536;     // uint16 block-relative indices

// One parameter tensor as the step kernel sees it.
struct TensorDesc {
  void* param;            // numel elements of the parameter dtype
  const void* grad;       // numel elements of the gradient dtype
  int64_t numel;
  int64_t first_block;    // global index of this tensor's block 0
  int64_t num_blocks;
  uint64_t ef_off;        // byte offsets into the state buffer
  uint64_t stats_off;
  uint64_t win_off;
  int32_t k_full;         // entries per window row, full block
  int32_t k_last;         // entries per window row, last block
};

// Threads per workgroup of the step kernel for a Top-K block of B_d elements
// (each thread owns 16 elements, so the block capacity is 16 * threads).
inline int threads_for_block(int block) { return block <= 1024 ? 64 : 256; }

// Per-launch scalars (passed by value as the kernel argument).
struct StepParams {
  const TensorDesc* tensors;
  const uint32_t* block_tensor;  // global block -> tensor index
  const float* wpow;             // [2 * kMaxWindow]: beta1^r, then beta2^r
  uint8_t* state;
  int64_t t;                     // step being taken (>= 1)
  int64_t total_blocks;
  int32_t n_tensors;
  int32_t block;                 // B_d
  int32_t bucket_log2;           // B_q = 1 << bucket_log2
  int32_t window;                // m
  int32_t n_old;                 // live rows written before step t: min(t, m) - 1
  int32_t new_slot;              // row slot written at step t: (t - 1) mod m
  int32_t k_full;                // entries per row of a full block (all tensors)
  int32_t decay_is_one;          // weight_decay * lr == 0
  float lr, decay, eps, c1, c2;
};

// Launchers (defined in microadam_kernels.hip).  Return hipSuccess or the
// launch error.
hipError_t launch_step(const StepParams& p, int param_bf16, int grad_bf16, int value_f32,
                       hipStream_t stream);

hipError_t launch_moments(const StepParams& p, int32_t tensor, int64_t first_block,
                          int64_t grid, float* mhat, float* vhat, int value_f32,
                          hipStream_t stream);

// Dynamic LDS bytes the step kernel needs for this configuration.
size_t step_lds_bytes(int block, int k_full, int value_f32);

}  // namespace microadam
