// Types shared by the host side of libmicroadam and its HIP kernels.
// Internal to the library: the public interface is include/microadam.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace microadam {

constexpr int kMaxWindow = 64;       // largest supported window m
constexpr int kMaxBlock = 65536;     // uint16 block-relative indices
constexpr int kSubBlockElems = 4096; // elements of a one-wave select block

// One parameter tensor as the kernels see it.  Its full blocks are the
// global blocks [first_block, first_block + num_full); a ragged last block
// (numel not a multiple of B_d) is numbered after every tensor's full blocks.
struct TensorDesc {
  void* param;            // numel elements of the parameter dtype
  const void* grad;       // numel elements of the gradient dtype
  int64_t numel;
  int64_t first_block;    // global number of block 0
  int64_t num_blocks;
  int64_t last_block;     // global number of block num_blocks - 1
  int32_t k_full;         // entries per window row, full block
  int32_t k_last;         // entries per window row, last block
  int32_t s_last;         // elements in the last block
  int32_t num_full;       // full blocks
  int64_t first_bucket;   // buckets spanning blocks: the tensor's bucket 0 in the table
  int64_t num_buckets;    // its buckets (0 with buckets inside blocks)
  int32_t ragged_before;  // tensors before this one that end in a ragged block
  int32_t reserved;
};

// Threads per workgroup for a Top-K block of B_d elements (each thread owns
// 16 elements, so the block capacity is 16 * threads).
inline int threads_for_block(int block) { return block <= 1024 ? 64 : 256; }

// State layout: three planes indexed by the global block number gb.
//   EF codes       ef_plane    + gb * B_d*b/8 (b = 4 or 8 bits per code)
//   (min, max)     stats_plane + gb * (B_d/B_q) * 8
//   window rows    win_plane   + gb * win_stride (m * k_full * entry_bytes
//                  rounded up to whole 128-byte lines)
// A block's window slot holds its m rows of k_q entries, row r at r*k_q.
// Global blocks [0, n_full) are full (B_d elements, k_full entries per row);
// blocks [n_full, total_blocks) are the ragged last blocks of tensors.
struct StepParams {
  const TensorDesc* tensors;
  const uint32_t* block_tensor;  // global block -> tensor index; NULL: found by binary search
  const float* wpow;             // [2 * kMaxWindow]: beta1^r, then beta2^r
  uint8_t* state;
  uint64_t ef_plane, stats_plane, win_plane;  // byte offsets into state
  uint64_t win_stride;           // bytes per block in the window plane (a multiple of 128)
  int64_t t;                     // step being taken (>= 1)
  int64_t total_blocks;
  int64_t n_full;                // full blocks (numbered first)
  int32_t block;                 // B_d
  int32_t bucket_log2;           // B_q = 1 << bucket_log2
  int32_t window;                // m
  int32_t n_live;                // rows live after step t: min(t, m)
  int32_t new_slot;              // row slot written at step t: (t - 1) mod m
  int32_t k_full;                // entries per row of a full block (all tensors)
  int32_t decay_is_one;          // weight_decay * lr == 0
  float lr, decay, eps, c1, c2;
  int32_t ef_mode;               // code format: bit 0 8-bit codes, bit 1 randomized rounding
  uint32_t seed_lo, seed_hi;     // key of the randomized rounding's stream
  // buckets spanning blocks (big_bucket = B_q > 0; else 0): the pairs of all
  // tensors' buckets in two tables of table_bytes at stats_plane (step t
  // fills table t mod 2), and per block two (min, max) partials at
  // partial_plane + gb * 16
  int64_t big_bucket;
  int64_t total_buckets;
  uint64_t table_bytes, partial_plane;
  int32_t n_tensors;
  // blocks above 4096 that are multiples of 4096, with buckets inside
  // blocks: device memory of the handle (NULL: the multi-wave select takes
  // every block) holding the threshold kernel's 128-byte per-block records,
  // then the list of the blocks it could not settle: their number (16
  // bytes) and the block numbers (4 bytes each), thr_list_bytes() in all
  uint8_t* thr;
};

// Bytes of the records and the list at StepParams::thr for `blocks` blocks.
__host__ __device__ inline size_t thr_list_offset(int64_t blocks) { return (size_t)blocks * 128; }
__host__ __device__ inline size_t thr_bytes(int64_t blocks) { return thr_list_offset(blocks) + 16 + (size_t)blocks * 4; }

// Steps with buckets spanning blocks: the per-block partials, their reduction
// into the new bucket table, and the quantization of the residual with it
// (k_span.hip).
hipError_t launch_select_partials(const StepParams& p, int grad_bf16, int value_f32, hipStream_t stream);
hipError_t launch_bucket_reduce(const StepParams& p, hipStream_t stream);
hipError_t launch_requant(const StepParams& p, int grad_bf16, int value_f32, hipStream_t stream);

// Launchers (microadam_launch.hip dispatches to the kernel translation
// units).  Return hipSuccess or the launch error.  Each takes the global
// blocks [first, first + count); the update of a block must follow its
// select, and blocks share nothing.
hipError_t launch_select(const StepParams& p, int grad_bf16, int value_f32, int64_t first, int64_t count,
                         hipStream_t stream);
hipError_t launch_update(const StepParams& p, int param_bf16, int value_f32, int64_t first, int64_t count,
                         hipStream_t stream);

hipError_t launch_moments(const StepParams& p, int64_t first_block, int64_t num_blocks,
                          float* mhat, float* vhat, int value_f32, hipStream_t stream);

// Dynamic LDS bytes the kernels need (the larger of the two step kernels).
size_t step_lds_bytes(int block, int k_full, int value_f32);

// Per translation unit: the one-wave select for blocks of up to 4096
// elements and the multi-wave select for larger blocks, in each
// error-feedback format (k_select_{near,rand}{4,8}.hip,
// k_select_large_{near,rand}{4,8}.hip), and the updates and moment exports
// (k_update.hip, k_update_large.hip).
hipError_t launch_select_near4(const StepParams& p, int grad_bf16, int value_f32, int64_t first, int64_t count,
                               hipStream_t stream);
hipError_t launch_select_near8(const StepParams& p, int grad_bf16, int value_f32, int64_t first, int64_t count,
                               hipStream_t stream);
hipError_t launch_select_rand4(const StepParams& p, int grad_bf16, int value_f32, int64_t first, int64_t count,
                               hipStream_t stream);
hipError_t launch_select_rand8(const StepParams& p, int grad_bf16, int value_f32, int64_t first, int64_t count,
                               hipStream_t stream);
hipError_t launch_select_large_near4(const StepParams& p, int grad_bf16, int value_f32, int64_t first, int64_t count,
                                  hipStream_t stream);
hipError_t launch_select_large_near8(const StepParams& p, int grad_bf16, int value_f32, int64_t first, int64_t count,
                                  hipStream_t stream);
hipError_t launch_select_large_rand4(const StepParams& p, int grad_bf16, int value_f32, int64_t first, int64_t count,
                                  hipStream_t stream);
hipError_t launch_select_large_rand8(const StepParams& p, int grad_bf16, int value_f32, int64_t first, int64_t count,
                                  hipStream_t stream);
hipError_t launch_update_blocks(const StepParams& p, int param_bf16, int value_f32, int64_t first, int64_t count,
                                hipStream_t stream);
hipError_t launch_update_large_blocks(const StepParams& p, int param_bf16, int value_f32, int64_t first,
                                      int64_t count, hipStream_t stream);
hipError_t launch_moments_blocks(const StepParams& p, int64_t first_block, int64_t num_blocks, float* mhat,
                                 float* vhat, int value_f32, hipStream_t stream);
hipError_t launch_moments_large_blocks(const StepParams& p, int64_t first_block, int64_t num_blocks, float* mhat,
                                       float* vhat, int value_f32, hipStream_t stream);
size_t update_lds_max(int nt);
size_t update_large_lds();

// The fused step (step_kernel.h, k_step_{near,rand}{4,8}.hip): every stage of
// a block in one workgroup, for blocks of 2049 to 4096 elements with at most
// kFusedMaxK entries per row, live rows of at most kFusedMaxChunks chunks of
// 64 entries, and parameters and gradients of one dtype (`bf16`).
constexpr int kFusedMaxK = 128;
constexpr int kFusedMaxChunks = 16;
hipError_t launch_step(const StepParams& p, int bf16, int value_f32, int64_t first, int64_t count,
                       hipStream_t stream);
hipError_t launch_step_near4(const StepParams& p, int bf16, int value_f32, int64_t first, int64_t count,
                             hipStream_t stream);
hipError_t launch_step_near8(const StepParams& p, int bf16, int value_f32, int64_t first, int64_t count,
                             hipStream_t stream);
hipError_t launch_step_rand4(const StepParams& p, int bf16, int value_f32, int64_t first, int64_t count,
                             hipStream_t stream);
hipError_t launch_step_rand8(const StepParams& p, int bf16, int value_f32, int64_t first, int64_t count,
                             hipStream_t stream);
size_t fused_lds_bytes(int value_f32);

}  // namespace microadam
