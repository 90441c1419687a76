/*
 * microadam.h -- C ABI of libmicroadam.so, a MicroAdam optimizer step for
 * AMD Instinct MI355X (gfx950).
 *
 * MicroAdam ("MicroAdam: Accurate Adaptive Optimization with Low Space
 * Overhead and Provable Convergence", Modoranu et al., 2024) keeps, per
 * parameter tensor:
 *   - a 4-bit error-feedback (EF) buffer e with per-bucket min/max metadata
 *     (delta, Delta) (Algorithm 1, the quantized EF; Section 3.1,
 *     "Quantization metadata");
 *   - a sliding window G = (I, V) of the last m sparse gradients, m rows of
 *     k block-relative uint16 indices and bf16 values (Section 3, notation;
 *     Section 3.1, "Top-K"; Section 3.2 for the 4-bytes-per-entry budget).
 * One step (Algorithm 1) decodes e and adds it to the gradient, keeps the
 * block-wise Top-K of |a| in a new window row, re-quantizes the residual
 * into e, rebuilds the Adam moments from the window (AdamStats, Algorithm 2)
 * and updates the parameters, with decoupled weight decay (Algorithm 4).
 *
 * Conventions for every call:
 *   - Return value: MICROADAM_OK (0) or a negative MICROADAM_ERR_* code.
 *     Arguments are validated before any device work is queued, so a call
 *     that fails leaves parameters and optimizer state untouched.
 *     microadam_error_string() names a code; microadam_last_error() gives the
 *     calling thread's most recent failure message in detail.
 *   - Device pointers are HIP device addresses owned by the caller.  Host
 *     pointers are plain host memory owned by the caller and only read
 *     during the call.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *     Device work is queued on it and the call returns without waiting.
 *   - A handle must be used by one host thread at a time.
 *   - No C++ exception crosses this interface.
 */
#ifndef MICROADAM_H
#define MICROADAM_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  MICROADAM_OK = 0,
  MICROADAM_ERR_INVALID_ARG = -1, /* null pointer, value out of range, misaligned buffer */
  MICROADAM_ERR_UNSUPPORTED = -2, /* a valid but unimplemented configuration */
  MICROADAM_ERR_SHAPE = -3,       /* tensor count or sizes differ from microadam_init */
  MICROADAM_ERR_STATE_SIZE = -4,  /* state buffer smaller than microadam_state_bytes */
  MICROADAM_ERR_HIP = -5,         /* a HIP runtime call failed (see microadam_last_error) */
  MICROADAM_ERR_NO_MEMORY = -6    /* host or library-internal allocation failed */
};

/* Element types of parameters and gradients. */
enum { MICROADAM_F32 = 0, MICROADAM_BF16 = 1 };

/*
 * Hyper-parameters, in the paper's notation (Section 3, notation; Appendix B
 * gives the values the paper trains with: density 0.01, m = 10, b = 4,
 * bucket 64, beta1 0.9, beta2 0.999, eps 1e-8).
 *
 *   density      k/d in (0, 1].  A Top-K block of s elements keeps
 *                k_s = min(s, max(1, ceil(density * s - 1e-9))) entries.
 *   beta1,beta2  moment decay rates in [0, 1).
 *   eps          added to sqrt(v-hat) in the update (Algorithm 1); > 0 (an
 *                element without window entries then takes a zero step).
 *   lr           default step size eta (microadam_step may override it).
 *   weight_decay lambda of the decoupled decay theta *= (1 - eta*lambda)
 *                (Algorithm 4); >= 0.
 *   window       m, rows in the sliding window, 1..64.
 *   ef_bits      b, bits per EF code: 4 (the paper's choice, Section 3.1) or
 *                8 (a wider code for the same buckets).
 *   ef_rounding  how Q rounds: MICROADAM_ROUND_NEAREST (Algorithm 2, half to
 *                even) or MICROADAM_ROUND_RANDOMIZED (Lemma 1: floor((x -
 *                delta)/u + xi), xi ~ U[0, 1), which makes Q unbiased).
 *   seed         key of the randomized rounding's random stream: element i
 *                of tensor j at step t draws xi = (w >> 8) * 2^-24 from word
 *                i mod 4 of Philox4x32-10 (Salmon et al., SC 2011) at counter
 *                (i/4 low word, i/4 high word, j, t) under the key (seed low
 *                word, seed high word); j is the tensor's position in the
 *                numels list of microadam_init.  The floor is taken of the
 *                exact sum.  Unused with NEAREST.
 *   ef_bucket    B_q, elements sharing one (delta, Delta) pair: a power of
 *                two in [8, 512] dividing topk_block (buckets inside blocks),
 *                or any size >= topk_block (buckets of each tensor's
 *                elements [c*B_q, (c+1)*B_q), spanning blocks; Section 3.1
 *                names 100K), which runs the quantization as a second pass
 *                over the block.
 *   topk_block   B_d, Top-K block size; at most
 *                65536 (block-relative indices are uint16).  This build
 *                implements multiples of 16 and returns
 *                MICROADAM_ERR_UNSUPPORTED for other valid sizes.
 *   window_value_dtype  MICROADAM_BF16 (the paper's choice, Section 3.2) or
 *                MICROADAM_F32 (lossless window values, for checking the
 *                moment rebuild).
 *   fused        0: every step runs a select kernel (EF decode, block Top-K,
 *                new row, re-quantization) and then an update kernel (moment
 *                rebuild, parameter update), the faster form on MI355X; 1:
 *                where the configuration allows (see microadam_step_kernels),
 *                all of a step in one fused kernel, one workgroup per block.
 *                Both give the same results.
 *   reserved     0.
 */
/* Rounding of the error-feedback quantizer. */
enum { MICROADAM_ROUND_NEAREST = 0, MICROADAM_ROUND_RANDOMIZED = 1 };

typedef struct microadam_config {
  double density;
  double beta1;
  double beta2;
  double eps;
  double lr;
  double weight_decay;
  int32_t window;
  int32_t ef_bits;
  int32_t ef_bucket;
  int32_t topk_block;
  int32_t window_value_dtype;
  int32_t ef_rounding;
  uint64_t seed;
  int32_t fused;
  int32_t reserved;
} microadam_config;

typedef struct microadam_handle_s* microadam_handle;

/*
 * Where one tensor's optimizer state lives inside the state buffer (byte
 * offsets from its start).  The buffer holds three planes, EF codes, bucket
 * stats and window, each starting 256-byte aligned.  In each plane every
 * Top-K block owns a record of fixed size, at plane + g * stride for its
 * global block number g.  Full blocks (B_d elements) are numbered first,
 * tensor by tensor, then the ragged last blocks of the tensors whose numel is
 * not a multiple of B_d; a ragged block's record is padded to full size.
 * Block q of a tensor has global number first_block + q, except its last
 * block (q = num_blocks - 1), whose number is last_block.
 *
 *   EF codes   B_d/2 bytes per block: element 2j of the block in the low
 *              nibble of byte j, element 2j+1 in the high nibble (nibbles
 *              past the block's elements are 0).  With ef_bits = 8, B_d
 *              bytes per block, element i in byte i.
 *   stats      B_d/B_q pairs of float32 (delta, Delta) per block = (min,
 *              max) of the bucket's residual; pair b covers the block's
 *              elements [b*B_q, (b+1)*B_q); pairs past its elements are
 *              unused.  With buckets spanning blocks (ef_bucket >= B_d and
 *              not a power of two in [8, 512] dividing B_d) the buckets are
 *              the tensor's elements [c*B_q, (c+1)*B_q), and their pairs
 *              live in two tables of bucket_table_bytes: the pair of bucket
 *              c written at step t is at stats_plane + (t mod 2) *
 *              bucket_table_bytes + 8*c (stats_stride is 0).  A plane of 16
 *              bytes per block of partial (min, max) pairs follows them.
 *   window     m*k_full*entry_bytes per block, rounded up to a multiple
 *              of 128 bytes (the stride): row r (the row written at
 *              step s is r = (s-1) mod m) starts at r*k_q*entry_bytes within
 *              the record and holds the block's k_q entries in ascending
 *              index order (k_q = k_last for the last block).  With bf16
 *              values an entry is one little-endian uint32 (index |
 *              bf16_bits << 16); with float32 values it is a uint32 index
 *              followed by the float32 value.  For B_d > 4096 the record
 *              continues, after the m rows (at byte m*k_full*entry_bytes),
 *              with a table of m*ceil(B_d/1024) uint32: entry (r, j) is the
 *              position in row r of the first entry whose index is at least
 *              1024*j (the entries of the block's 1024-element quarter j
 *              are the positions [entry (r, j), entry (r, j+1)), the last
 *              ending at k_q).
 */
typedef struct microadam_layout {
  int64_t numel;
  int64_t num_blocks;
  int64_t num_buckets;
  int32_t k_full;      /* entries per row of a full block */
  int32_t k_last;      /* entries per row of the last block */
  int32_t entry_bytes; /* 4 (bf16 values) or 8 (float32 values) */
  int32_t reserved;
  int64_t first_block; /* global number of block 0 */
  int64_t last_block;  /* global number of block num_blocks - 1 */
  uint64_t ef_plane, ef_stride;
  uint64_t stats_plane, stats_stride;
  uint64_t window_plane, window_stride;
  uint64_t bucket_table_bytes; /* buckets spanning blocks: see stats above; else 0 */
} microadam_layout;

/*
 * Size in bytes of the device state buffer for tensors of the given element
 * counts (numels[0..n_tensors), each >= 1).  Pure host computation: per
 * Top-K block B_d/2 bytes of EF codes, 8*B_d/B_q bytes of bucket stats and
 * m*k_full*entry_bytes of window rounded up to 128 bytes, each plane
 * 256-byte aligned.  This is the
 * paper's 0.5d + 4mk (Section 3.2) plus the (delta, Delta) metadata of
 * Section 3.1, per-block rounding of k and the padding of each tensor's last
 * block.
 */
int microadam_state_bytes(const microadam_config* cfg, const int64_t* numels,
                          int32_t n_tensors, uint64_t* out_bytes);

/*
 * Creates a handle for the tensor list numels[0..n_tensors) and clears the
 * caller-owned device buffer `state` (>= microadam_state_bytes bytes, 256-byte
 * aligned) on `stream`: e = 0, delta = Delta = 0 as in the initialisation of
 * Algorithm 1.  The step counter starts at 0 (the next step is t = 1).
 * param_dtype / grad_dtype: MICROADAM_F32 or MICROADAM_BF16.
 * The library keeps small device tables of its own (freed by destroy:
 * the block -> tensor table, the window weights, and with Top-K blocks above
 * 4096 elements that are multiples of 4096 a 128-byte record per block
 * and a list of the blocks the threshold pass could not settle, 4 bytes per
 * block);
 * `state` stays owned by the caller and must outlive the handle.
 */
int microadam_init(const microadam_config* cfg, const int64_t* numels,
                   int32_t n_tensors, int32_t param_dtype, int32_t grad_dtype,
                   void* state, uint64_t state_bytes, void* stream,
                   microadam_handle* out);

/*
 * One MicroAdam step (Algorithm 1 with the decay of Algorithm 4) over all
 * tensors, queued on `stream` (microadam_step_kernels launches).  params[j] (updated in place)
 * and grads[j] (read only) are device pointers to numels[j] contiguous
 * elements of the init dtypes, 16-byte aligned.  lr: the step size eta for
 * this step, or NaN to use cfg.lr.  The step counter t advances by one.
 * Non-finite gradients (NaN, +-inf), which the method leaves undefined, give
 * unspecified parameters and state in the Top-K blocks that hold them (in
 * their buckets, when buckets span blocks); every other block is computed as
 * if they were absent, and no memory outside params, grads and the state is
 * touched.
 */
int microadam_step(microadam_handle h, void* const* params,
                   const void* const* grads, int32_t n_tensors, double lr,
                   void* stream);

/* Frees the handle and the library's device table (waits for nothing;
 * the caller must not destroy a handle whose step may still be running on
 * a stream it will not synchronize).  NULL is accepted. */
int microadam_destroy(microadam_handle h);

/* Steps taken so far (the t of the last step), or a negative error code. */
int64_t microadam_get_step(microadam_handle h);

/* Sets the step counter, e.g. after restoring a saved state buffer: the next
 * step is t + 1.  t >= 0. */
int microadam_set_step(microadam_handle h, int64_t t);

/* Layout of tensor `tensor`'s state (see microadam_layout). */
int microadam_tensor_layout(microadam_handle h, int32_t tensor,
                            microadam_layout* out);

/*
 * Test support: recomputes the dense float32 m-hat and v-hat of tensor
 * `tensor` from the window as it stands after the last step (AdamStats,
 * Algorithm 2, at the current t >= 1), into device buffers of numel floats.
 */
int microadam_debug_moments(microadam_handle h, int32_t tensor, float* mhat,
                            float* vhat, void* stream);

/*
 * Kernel launches per microadam_step (fixed at init), or a negative error
 * code: 1 where the step runs as one fused kernel (cfg.fused = 1, Top-K
 * blocks of 2049 to 4096 elements, at most 128 entries per row, m *
 * ceil(k/64) <= 16, parameters and gradients of one dtype, buckets inside
 * blocks); 2 (select, then update) otherwise; 4 with buckets spanning blocks
 * (select, bucket reduction, quantization, update); 4 with Top-K blocks
 * above 4096 elements that are multiples of 4096 and buckets inside blocks
 * (a threshold pass over each block, the select of its 4096-element
 * sub-blocks, the multi-wave select of the blocks whose threshold the first
 * pass left open, update).
 */
int microadam_step_kernels(microadam_handle h);

/*
 * Profiling.  With profiling on (off after init), every microadam_step
 * records HIP events on its stream around its kernels.  Events are
 * created on the first call that turns profiling on, with the init device
 * current.  Every call that turns it on starts a new total for
 * microadam_kernel_times_total.
 */
int microadam_set_profiling(microadam_handle h, int32_t on);

/*
 * Durations in milliseconds of the kernels of the last step, which must have
 * been taken with profiling on: out_ms[0] = select (EF decode, block Top-K,
 * new window row, EF re-quantisation), out_ms[1] = update (moment rebuild
 * from the window and parameter update); for a fused step (see
 * microadam_step_kernels) out_ms[0] is the fused kernel and out_ms[1] is 0.  Blocks until that step is done.
 * out_ms: 2 host floats.
 */
int microadam_kernel_times(microadam_handle h, float* out_ms);

/*
 * Summed kernel durations of every step profiled since profiling was last
 * switched on (or since the previous call of this function), without
 * synchronizing between steps: out_ms[0] = select, out_ms[1] = update, in
 * milliseconds (summed as microadam_kernel_times reports one step), and
 * *out_steps = the number of steps they cover; the totals then restart at 0.
 * The library keeps each profiled step's events in a ring of four sets and
 * reads a set when it is needed again, four profiled steps later.  Blocks
 * until the steps counted are done.  out_ms: 2 host floats; out_steps: one
 * host int64.  Errors: MICROADAM_ERR_INVALID_ARG for NULL outputs.
 */
int microadam_kernel_times_total(microadam_handle h, float* out_ms, int64_t* out_steps);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): step t
 * (>= 1) of the tensor list numels[0..n_tensors) on a caller-owned state
 * buffer laid out as microadam_init lays it out for the same cfg and numels
 * (>= microadam_state_bytes bytes, 256-byte aligned), holding the state
 * after step t - 1: all zero bytes before step 1, which the caller provides.
 * No handle is used and nothing is allocated: the tensor table and window
 * weights go to a static device array of the library, at most 4096 tensors
 * (393 KB; every GPU the library runs on holds its own copy until the
 * process ends), and the kernels are those of microadam_step, with the same
 * results.  params, grads, lr, stream as for microadam_step; param_dtype and
 * grad_dtype as for microadam_init.  Calls that overlap on one GPU (other
 * streams, other host threads) race on the shared array, and each call
 * overwrites what the last one left there; calls on one stream are ordered.
 * Errors: MICROADAM_ERR_UNSUPPORTED for more than 4096 tensors, else those
 * of microadam_init and microadam_step; nothing is queued on failure.
 */
int microadam_step_noalloc(const microadam_config* cfg, const int64_t* numels, int32_t n_tensors,
                           int32_t param_dtype, int32_t grad_dtype, void* state, uint64_t state_bytes,
                           int64_t t, void* const* params, const void* const* grads, double lr,
                           void* stream);

const char* microadam_error_string(int code);

/* The calling thread's most recent error message ("" if none). */
const char* microadam_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* MICROADAM_H */
