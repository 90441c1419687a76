// Host side of libmicroadam: configuration checks, the state layout planner,
// the device descriptor tables and the per-step constants.  Every entry point
// validates its arguments before queueing device work.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstddef>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "microadam.h"
#include "microadam_device.h"

using microadam::StepParams;
using microadam::TensorDesc;

namespace {

// The calling thread's last error message, in a fixed buffer (reporting an
// error allocates nothing).
thread_local char g_last_error[512];

int fail(int code, const char* msg) {
  std::snprintf(g_last_error, sizeof(g_last_error), "%s", msg);
  return code;
}

int hip_fail(hipError_t e, const char* what) {
  std::snprintf(g_last_error, sizeof(g_last_error), "%s: %s", what, hipGetErrorString(e));
  return MICROADAM_ERR_HIP;
}

void clear_error() { g_last_error[0] = '\0'; }

constexpr uint64_t kAlign = 256;
constexpr size_t kMaxLds = 65536;        // dynamic LDS budget per workgroup

uint64_t align_up(uint64_t x) { return (x + kAlign - 1) & ~(kAlign - 1); }

// k for a block of s elements: ceil(density * s), clamped to [1, s]; the
// 1e-9 guard keeps products such as 0.01 * 100 from rounding up to 2.
int64_t block_k(int64_t s, double density) {
  int64_t k = (int64_t)std::ceil(density * (double)s - 1e-9);
  if (k < 1) k = 1;
  if (k > s) k = s;
  return k;
}

bool is_pow2(int64_t x) { return x > 0 && (x & (x - 1)) == 0; }

// Buckets of B_q >= B_d elements that are not the block-local kind (a power
// of two in [8, 512] dividing B_d): each tensor's buckets restart at its
// element 0, so a bucket may hold several blocks and a block may straddle two.
bool buckets_span_blocks(const microadam_config* c) {
  const bool local = is_pow2(c->ef_bucket) && c->ef_bucket >= 8 && c->ef_bucket <= 512 && c->topk_block > 0 &&
                     c->topk_block % c->ef_bucket == 0;
  return !local && c->ef_bucket >= c->topk_block;
}

int validate_config(const microadam_config* c) {
  if (!c) return fail(MICROADAM_ERR_INVALID_ARG, "config is NULL");
  if (!(c->density > 0.0 && c->density <= 1.0))
    return fail(MICROADAM_ERR_INVALID_ARG, "density must be in (0, 1]");
  if (!(c->beta1 >= 0.0 && c->beta1 < 1.0) || !(c->beta2 >= 0.0 && c->beta2 < 1.0))
    return fail(MICROADAM_ERR_INVALID_ARG, "beta1 and beta2 must be in [0, 1)");
  if (!(c->eps > 0.0) || !std::isfinite(c->eps))
    return fail(MICROADAM_ERR_INVALID_ARG, "eps must be finite and > 0");
  if (!std::isfinite(c->lr)) return fail(MICROADAM_ERR_INVALID_ARG, "lr must be finite");
  if (!(c->weight_decay >= 0.0) || !std::isfinite(c->weight_decay))
    return fail(MICROADAM_ERR_INVALID_ARG, "weight_decay must be finite and >= 0");
  if (c->window < 1) return fail(MICROADAM_ERR_INVALID_ARG, "window must be >= 1");
  if (c->window > microadam::kMaxWindow)
    return fail(MICROADAM_ERR_UNSUPPORTED, "window above 64 is not supported");
  if (c->ef_bits < 1 || c->ef_bits > 16) return fail(MICROADAM_ERR_INVALID_ARG, "ef_bits out of range");
  if (c->ef_bits != 4 && c->ef_bits != 8) return fail(MICROADAM_ERR_UNSUPPORTED, "ef_bits must be 4 or 8");
  if (c->ef_bucket < 2) return fail(MICROADAM_ERR_INVALID_ARG, "ef_bucket must be >= 2");
  if (c->topk_block < 1) return fail(MICROADAM_ERR_INVALID_ARG, "topk_block must be >= 1");
  if (c->topk_block > microadam::kMaxBlock)
    return fail(MICROADAM_ERR_UNSUPPORTED, "topk_block above 65536 does not fit uint16 indices");
  if (!buckets_span_blocks(c)) {
    if (!is_pow2(c->ef_bucket) || c->ef_bucket < 8 || c->ef_bucket > 512)
      return fail(MICROADAM_ERR_UNSUPPORTED, "ef_bucket must be a power of two in [8, 512], or >= topk_block");
    if (c->topk_block % c->ef_bucket != 0)
      return fail(MICROADAM_ERR_INVALID_ARG, "topk_block must be a multiple of ef_bucket");
  }
  if (c->topk_block % 16 != 0)
    return fail(MICROADAM_ERR_UNSUPPORTED, "topk_block must be a multiple of 16");
  if (c->window_value_dtype != MICROADAM_BF16 && c->window_value_dtype != MICROADAM_F32)
    return fail(MICROADAM_ERR_INVALID_ARG, "window_value_dtype must be BF16 or F32");
  if (c->ef_rounding != MICROADAM_ROUND_NEAREST && c->ef_rounding != MICROADAM_ROUND_RANDOMIZED)
    return fail(MICROADAM_ERR_INVALID_ARG, "ef_rounding must be NEAREST or RANDOMIZED");
  if (c->fused != 0 && c->fused != 1) return fail(MICROADAM_ERR_INVALID_ARG, "fused must be 0 or 1");
  if (c->reserved != 0) return fail(MICROADAM_ERR_INVALID_ARG, "reserved must be 0");
  return MICROADAM_OK;
}

struct TensorPlan {
  int64_t numel, num_blocks, num_buckets, num_full, first_block, last_block;
  int64_t first_bucket;  // buckets spanning blocks: bucket 0's place in the tables
  int32_t k_full, k_last, s_last;
  int32_t ragged_before;  // tensors before this one that end in a ragged block
};

// Byte offsets of the three state planes; every block owns a record of fixed
// size in each, addressed by its global block number.
struct Planes {
  uint64_t ef, stats, win, total;
  uint64_t ef_stride, stats_stride, win_stride;  // bytes per block
  int64_t n_full, n_blocks;
  // buckets spanning blocks: two tables of n_buckets (delta, Delta) pairs
  // (table_bytes each) in the stats plane, and a partials plane of 16 bytes
  // per block
  bool big = false;
  int64_t n_buckets = 0;
  uint64_t table_bytes = 0, partial = 0;
};

int entry_bytes(const microadam_config* c) { return c->window_value_dtype == MICROADAM_F32 ? 8 : 4; }

// Full blocks are numbered first, tensor by tensor; the ragged last blocks
// follow, so that the full blocks form one range of equal blocks.
// out: n entries (host memory of the caller; nothing is allocated here).
int make_plan(const microadam_config* c, const int64_t* numels, int32_t n, TensorPlan* out, Planes& pl) {
  if (n < 1) return fail(MICROADAM_ERR_INVALID_ARG, "n_tensors must be >= 1");
  if (!numels) return fail(MICROADAM_ERR_INVALID_ARG, "numels is NULL");
  const int64_t B = c->topk_block, Bq = c->ef_bucket, m = c->window;
  const int64_t eb = entry_bytes(c);
  const int32_t k_full = (int32_t)block_k(B, c->density);
  pl.big = buckets_span_blocks(c);
  pl.n_buckets = 0;
  pl.ef_stride = (uint64_t)B * (uint64_t)c->ef_bits / 8;
  pl.stats_stride = pl.big ? 0 : (uint64_t)(B / Bq) * 8;
  // whole 128-byte lines per record, so that a row can be written as whole
  // lines without touching another block's record; blocks above 4096 add a
  // table of m * ceil(B_d/1024) uint32 segment starts behind the rows
  const uint64_t table = B > 4096 ? (uint64_t)m * ((B + 1023) / 1024) * 4 : 0;
  pl.win_stride = ((uint64_t)m * k_full * eb + table + 127) & ~(uint64_t)127;
  int64_t full = 0;
  for (int32_t j = 0; j < n; ++j) {
    const int64_t d = numels[j];
    if (d < 1) return fail(MICROADAM_ERR_INVALID_ARG, "every numel must be >= 1");
    if (d > ((int64_t)1 << 50)) return fail(MICROADAM_ERR_INVALID_ARG, "numel too large");
    TensorPlan p;
    p.numel = d;
    p.num_blocks = (d + B - 1) / B;
    p.num_buckets = (d + Bq - 1) / Bq;
    p.num_full = d / B;
    p.first_block = full;
    p.k_full = k_full;
    p.s_last = (int32_t)(d - (p.num_blocks - 1) * B);
    p.k_last = (int32_t)block_k(p.s_last, c->density);
    p.first_bucket = pl.big ? pl.n_buckets : 0;
    if (pl.big) pl.n_buckets += p.num_buckets;
    full += p.num_full;
    out[j] = p;
  }
  int64_t next = full;
  for (int32_t j = 0; j < n; ++j) {
    TensorPlan& p = out[j];
    p.ragged_before = (int32_t)(next - full);
    p.last_block = p.num_full < p.num_blocks ? next++ : p.first_block + p.num_blocks - 1;
  }
  const uint64_t nb = (uint64_t)next;
  pl.n_full = full;
  pl.n_blocks = next;
  pl.ef = 0;
  pl.stats = align_up(pl.ef + nb * pl.ef_stride);
  if (pl.big) {
    pl.table_bytes = (uint64_t)pl.n_buckets * 8;
    pl.partial = align_up(pl.stats + 2 * pl.table_bytes);
    pl.win = align_up(pl.partial + nb * 16);
  } else {
    pl.win = align_up(pl.stats + nb * pl.stats_stride);
  }
  pl.total = align_up(pl.win + nb * pl.win_stride);
  return MICROADAM_OK;
}

using microadam::threads_for_block;

// Launch limits of a plan (blocks per launch; buckets spanning blocks).
int check_launch_size(const microadam_config* cfg, const Planes& pl) {
  const int64_t total_blocks = pl.n_blocks;
  const int nt = threads_for_block(cfg->topk_block);
  if (total_blocks * (int64_t)nt >= ((int64_t)1 << 32) || total_blocks >= ((int64_t)1 << 31))
    return fail(MICROADAM_ERR_UNSUPPORTED, "too many Top-K blocks for one launch");
  if (pl.big && (total_blocks >= ((int64_t)1 << 28) || pl.table_bytes >= ((uint64_t)1 << 32)))
    return fail(MICROADAM_ERR_UNSUPPORTED, "too many blocks or buckets for buckets spanning blocks");
  return MICROADAM_OK;
}

// One fused kernel per step when asked for and where a block fits one
// 256-thread workgroup and its new row and live rows fit the kernel's LDS;
// else a select and an update kernel (or four launches with buckets
// spanning blocks).
bool use_fused(const microadam_config* cfg, const Planes& pl, int32_t k_full, int32_t param_bf16,
               int32_t grad_bf16) {
  const int32_t parts = (k_full + 63) / 64;
  return cfg->fused == 1 && !pl.big && cfg->topk_block > 2048 && cfg->topk_block <= 4096 &&
         k_full <= microadam::kFusedMaxK && cfg->window * parts <= microadam::kFusedMaxChunks &&
         param_bf16 == grad_bf16;
}

int32_t bucket_log2_of(const microadam_config* cfg, const Planes& pl) {
  int32_t b = 0;
  if (!pl.big)
    while ((1 << b) < cfg->ef_bucket) ++b;
  return b;
}

// The kernels' view of tensor j (the param and grad addresses are set per step).
TensorDesc desc_of(const TensorPlan& p, const Planes& pl) {
  TensorDesc d;
  std::memset(&d, 0, sizeof(d));
  d.numel = p.numel;
  d.first_block = p.first_block;
  d.num_blocks = p.num_blocks;
  d.last_block = p.last_block;
  d.k_full = p.k_full;
  d.k_last = p.k_last;
  d.s_last = p.s_last;
  d.num_full = (int32_t)p.num_full;
  d.first_bucket = p.first_bucket;
  d.num_buckets = pl.big ? p.num_buckets : 0;
  d.ragged_before = p.ragged_before;
  return d;
}

// beta1^r and beta2^r, r < m, from binary64 rounded once (Algorithm 2).
void window_weights(const microadam_config* cfg, float* w) {
  for (int r = 0; r < 2 * microadam::kMaxWindow; ++r) w[r] = 0.0f;
  for (int r = 0; r < cfg->window; ++r) {
    w[r] = (float)std::pow(cfg->beta1, (double)r);
    w[microadam::kMaxWindow + r] = (float)std::pow(cfg->beta2, (double)r);
  }
}

// Per-step constants, derived in binary64 and rounded once to binary32: the
// bias corrections (1 - beta)/(1 - beta^t) of AdamStats (Algorithm 2) and the
// decay factor 1 - eta*lambda (Algorithm 4).  The window weights beta^r live
// in a device table (`wpow`).
void fill_step_params(const microadam_config& c, const Planes& pl, int32_t k_full, int32_t n_tensors,
                      int32_t bucket_log2, int64_t t, double lr, const TensorDesc* tensors,
                      const uint32_t* block_tensor, const float* wpow, uint8_t* state, StepParams& p) {
  const int m = c.window;
  std::memset(&p, 0, sizeof(p));
  p.tensors = tensors;
  p.block_tensor = block_tensor;
  p.wpow = wpow;
  p.state = state;
  p.ef_plane = pl.ef;
  p.stats_plane = pl.stats;
  p.win_plane = pl.win;
  p.win_stride = pl.win_stride;
  p.t = t;
  p.total_blocks = pl.n_blocks;
  p.n_full = pl.n_full;
  p.block = c.topk_block;
  p.bucket_log2 = bucket_log2;
  p.window = m;
  p.n_live = (int32_t)(t < m ? t : m);
  p.new_slot = (int32_t)((t - 1) % m);
  p.k_full = k_full;
  p.lr = (float)lr;
  p.decay = (float)(1.0 - lr * c.weight_decay);
  p.decay_is_one = (lr * c.weight_decay == 0.0) ? 1 : 0;
  p.eps = (float)c.eps;
  p.c1 = (float)((1.0 - c.beta1) / (1.0 - std::pow(c.beta1, (double)t)));
  p.c2 = (float)((1.0 - c.beta2) / (1.0 - std::pow(c.beta2, (double)t)));
  p.ef_mode = (c.ef_bits == 8 ? 1 : 0) | (c.ef_rounding == MICROADAM_ROUND_RANDOMIZED ? 2 : 0);
  p.seed_lo = (uint32_t)c.seed;
  p.seed_hi = (uint32_t)(c.seed >> 32);
  if (pl.big) {
    p.big_bucket = c.ef_bucket;
    p.total_buckets = pl.n_buckets;
    p.table_bytes = pl.table_bytes;
    p.partial_plane = pl.partial;
  }
  p.n_tensors = n_tensors;
}

// Queues the launches of one step on `s`; rec(i) records profiling event i
// (0: start, 1, 2: between the select and the update, 3: end).
template <typename Rec>
int queue_step(const StepParams& p, bool fused, bool big, int32_t param_bf16, int32_t grad_bf16,
               int32_t value_f32, hipStream_t s, Rec rec) {
  hipError_t e;
  if ((e = rec(0)) != hipSuccess) return hip_fail(e, "hipEventRecord");
  if (fused) {
    e = microadam::launch_step(p, param_bf16, value_f32, 0, p.total_blocks, s);
    if (e != hipSuccess) return hip_fail(e, "launching the step kernel");
  } else if (big) {
    // select with per-block partials, the bucket reduction, the quantization
    // of the residual
    e = microadam::launch_select_partials(p, grad_bf16, value_f32, s);
    if (e != hipSuccess) return hip_fail(e, "launching the select kernel");
    e = microadam::launch_bucket_reduce(p, s);
    if (e != hipSuccess) return hip_fail(e, "launching the bucket reduction");
    e = microadam::launch_requant(p, grad_bf16, value_f32, s);
    if (e != hipSuccess) return hip_fail(e, "launching the quantization kernel");
  } else {
    e = microadam::launch_select(p, grad_bf16, value_f32, 0, p.total_blocks, s);
    if (e != hipSuccess) return hip_fail(e, "launching the select kernel");
  }
  if ((e = rec(1)) != hipSuccess || (e = rec(2)) != hipSuccess) return hip_fail(e, "hipEventRecord");
  if (!fused) {
    e = microadam::launch_update(p, param_bf16, value_f32, 0, p.total_blocks, s);
    if (e != hipSuccess) return hip_fail(e, "launching the update kernel");
  }
  if ((e = rec(3)) != hipSuccess) return hip_fail(e, "hipEventRecord");
  return MICROADAM_OK;
}

}  // namespace

// A device copy of the tensor table for one set of param/grad addresses.
// Callers that alternate between a few gradient buffers reuse their tables
// instead of uploading one per step.
struct TableSlot {
  TensorDesc* d = nullptr;          // device table
  TensorDesc* h = nullptr;          // pinned host staging of the same table
  hipEvent_t upload_done = nullptr; // the last upload from `h` has finished
  uint64_t last_use = 0;            // 0: never filled
};

constexpr int kTableSlots = 4;

struct microadam_handle_s {
  microadam_config cfg;
  std::vector<TensorPlan> plans;
  Planes planes;
  int32_t param_bf16 = 0, grad_bf16 = 0, value_f32 = 0;
  int32_t bucket_log2 = 0;
  bool fused = false;                 // steps run as the one fused kernel
  uint8_t* state = nullptr;
  uint64_t state_bytes = 0;
  int64_t t = 0;
  int64_t total_blocks = 0;
  int device = 0;
  uint32_t* d_block_tensor = nullptr; // device: global block -> tensor
  float* d_wpow = nullptr;            // device: beta1^r, beta2^r for r < 64
  uint8_t* d_thr = nullptr;           // device: the threshold kernel's per-block records, or NULL
  TableSlot slots[kTableSlots];
  uint64_t use_clock = 0;
  int current = -1;                   // slot used by the last step
  hipEvent_t step_done = nullptr;     // last launch of this handle finished
  bool profiling = false;
  bool timed = false;                 // the last step recorded events
  // A ring of event sets for the profiled steps: select start, select end,
  // update start, update end.  A set holds a step whose durations are not
  // yet in the totals while pending[slot] is set.
  static constexpr int kProfSlots = 4;
  hipEvent_t ev[kProfSlots][4] = {};
  bool pending[kProfSlots] = {};
  int32_t prof_slot = 0;              // set of the last profiled step
  int64_t prof_count = 0;             // profiled steps since profiling was switched on
  double total_ms[2] = {0.0, 0.0};    // summed durations of the steps folded so far
  int64_t total_steps = 0;
};

namespace {

void release(microadam_handle h) {
  if (!h) return;
  if (h->step_done) {
    (void)hipEventSynchronize(h->step_done);
    (void)hipEventDestroy(h->step_done);
  }
  for (TableSlot& t : h->slots) {
    if (t.upload_done) {
      (void)hipEventSynchronize(t.upload_done);
      (void)hipEventDestroy(t.upload_done);
    }
    if (t.d) (void)hipFree(t.d);
    if (t.h) (void)hipHostFree(t.h);
  }
  for (auto& set : h->ev)
    for (hipEvent_t& e : set)
      if (e) (void)hipEventDestroy(e);
  if (h->d_block_tensor) (void)hipFree(h->d_block_tensor);
  if (h->d_wpow) (void)hipFree(h->d_wpow);
  if (h->d_thr) (void)hipFree(h->d_thr);
  delete h;
}

// Durations of the step recorded in event set `slot` (select, update),
// waiting for them.
hipError_t slot_times(microadam_handle h, int slot, float* out_ms) {
  hipError_t e;
  const hipEvent_t* ev = h->ev[slot];
  out_ms[0] = out_ms[1] = 0.0f;
  if ((e = hipEventSynchronize(ev[1])) != hipSuccess || (e = hipEventSynchronize(ev[3])) != hipSuccess ||
      (e = hipEventElapsedTime(&out_ms[0], ev[0], ev[1])) != hipSuccess ||
      (e = hipEventElapsedTime(&out_ms[1], ev[2], ev[3])) != hipSuccess)
    return e;
  return hipSuccess;
}

// Adds the durations of the step pending in event set `slot` to the totals.
hipError_t fold_slot(microadam_handle h, int slot) {
  if (!h->pending[slot]) return hipSuccess;
  float ms[2];
  const hipError_t e = slot_times(h, slot, ms);
  if (e != hipSuccess) return e;
  h->total_ms[0] += ms[0];
  h->total_ms[1] += ms[1];
  ++h->total_steps;
  h->pending[slot] = false;
  return hipSuccess;
}

// Per-step constants of a handle's step t.
void fill_constants(const microadam_handle h, int64_t t, double lr, StepParams& p) {
  fill_step_params(h->cfg, h->planes, h->plans.empty() ? 0 : h->plans[0].k_full, (int32_t)h->plans.size(),
                   h->bucket_log2, t, lr, h->current >= 0 ? h->slots[h->current].d : nullptr, h->d_block_tensor,
                   h->d_wpow, h->state, p);
  p.thr = h->d_thr;
}

int check_handle(microadam_handle h) {
  if (!h) return fail(MICROADAM_ERR_INVALID_ARG, "handle is NULL");
  return MICROADAM_OK;
}

int check_device(microadam_handle h) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev != h->device)
    return fail(MICROADAM_ERR_INVALID_ARG, "the current device differs from the one at init");
  return MICROADAM_OK;
}

}  // namespace

extern "C" {

int microadam_state_bytes(const microadam_config* cfg, const int64_t* numels, int32_t n_tensors,
                          uint64_t* out_bytes) {
  if (!out_bytes) return fail(MICROADAM_ERR_INVALID_ARG, "out_bytes is NULL");
  int rc = validate_config(cfg);
  if (rc) return rc;
  if (n_tensors < 1) return fail(MICROADAM_ERR_INVALID_ARG, "n_tensors must be >= 1");
  std::vector<TensorPlan> plans((size_t)n_tensors);
  Planes pl;
  rc = make_plan(cfg, numels, n_tensors, plans.data(), pl);
  if (rc) return rc;
  *out_bytes = pl.total;
  return MICROADAM_OK;
}

int microadam_init(const microadam_config* cfg, const int64_t* numels, int32_t n_tensors,
                   int32_t param_dtype, int32_t grad_dtype, void* state, uint64_t state_bytes,
                   void* stream, microadam_handle* out) {
  if (!out) return fail(MICROADAM_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  int rc = validate_config(cfg);
  if (rc) return rc;
  if ((param_dtype != MICROADAM_F32 && param_dtype != MICROADAM_BF16) ||
      (grad_dtype != MICROADAM_F32 && grad_dtype != MICROADAM_BF16))
    return fail(MICROADAM_ERR_INVALID_ARG, "param_dtype / grad_dtype must be F32 or BF16");
  if (n_tensors < 1) return fail(MICROADAM_ERR_INVALID_ARG, "n_tensors must be >= 1");
  std::vector<TensorPlan> plans((size_t)n_tensors);
  Planes pl;
  rc = make_plan(cfg, numels, n_tensors, plans.data(), pl);
  if (rc) return rc;
  const uint64_t total = pl.total;
  if (!state) return fail(MICROADAM_ERR_INVALID_ARG, "state is NULL");
  if ((uintptr_t)state % kAlign) return fail(MICROADAM_ERR_INVALID_ARG, "state must be 256-byte aligned");
  if (state_bytes < total)
    return fail(MICROADAM_ERR_STATE_SIZE, "state buffer smaller than microadam_state_bytes");
  rc = check_launch_size(cfg, pl);
  if (rc) return rc;
  const int64_t total_blocks = pl.n_blocks;

  microadam_handle h = new (std::nothrow) microadam_handle_s;
  if (!h) return fail(MICROADAM_ERR_NO_MEMORY, "handle allocation failed");
  h->cfg = *cfg;
  h->plans = std::move(plans);
  h->planes = pl;
  h->param_bf16 = param_dtype == MICROADAM_BF16;
  h->grad_bf16 = grad_dtype == MICROADAM_BF16;
  h->value_f32 = cfg->window_value_dtype == MICROADAM_F32;
  h->bucket_log2 = bucket_log2_of(cfg, pl);
  h->state = (uint8_t*)state;
  h->state_bytes = state_bytes;
  h->total_blocks = total_blocks;

  if (microadam::step_lds_bytes(cfg->topk_block, h->plans[0].k_full, h->value_f32) > kMaxLds) {
    release(h);
    return fail(MICROADAM_ERR_UNSUPPORTED, "k per block too large for the LDS budget");
  }
  h->fused = use_fused(cfg, pl, h->plans[0].k_full, h->param_bf16, h->grad_bf16);

  hipError_t e = hipGetDevice(&h->device);
  if (e != hipSuccess) { release(h); return hip_fail(e, "hipGetDevice"); }
  const size_t nd = h->plans.size();
  if ((e = hipMalloc((void**)&h->d_block_tensor, (size_t)total_blocks * 4)) != hipSuccess ||
      (e = hipMalloc((void**)&h->d_wpow, 2 * microadam::kMaxWindow * sizeof(float))) != hipSuccess ||
      (e = hipEventCreateWithFlags(&h->step_done, hipEventDisableTiming)) != hipSuccess) {
    release(h);
    return hip_fail(e, "allocating the block table");
  }
  // blocks above 4096 that are multiples of 4096, buckets inside blocks:
  // the threshold kernel's records (128 bytes per block, written every step)
  // and its list of unsettled blocks, whose count starts at 0 (the update
  // kernel clears it after every step)
  if (cfg->topk_block > microadam::kSubBlockElems && cfg->topk_block % microadam::kSubBlockElems == 0 &&
      !h->planes.big && !h->fused) {
    if ((e = hipMalloc((void**)&h->d_thr, microadam::thr_bytes(total_blocks))) != hipSuccess ||
        (e = hipMemset(h->d_thr + microadam::thr_list_offset(total_blocks), 0, 16)) != hipSuccess) {
      release(h);
      return hip_fail(e, "allocating the threshold records");
    }
  }
  {
    float w[2 * microadam::kMaxWindow];
    window_weights(cfg, w);
    if ((e = hipMemcpy(h->d_wpow, w, sizeof(w), hipMemcpyHostToDevice)) != hipSuccess) {
      release(h);
      return hip_fail(e, "uploading the window weights");
    }
  }
  for (TableSlot& t : h->slots) {
    if ((e = hipMalloc((void**)&t.d, nd * sizeof(TensorDesc))) != hipSuccess ||
        (e = hipHostMalloc((void**)&t.h, nd * sizeof(TensorDesc), hipHostMallocDefault)) != hipSuccess ||
        (e = hipEventCreateWithFlags(&t.upload_done, hipEventDisableTiming)) != hipSuccess) {
      release(h);
      return hip_fail(e, "allocating the descriptor tables");
    }
  }
  std::vector<uint32_t> bt((size_t)total_blocks);
  for (size_t j = 0; j < nd; ++j) {
    const TensorPlan& p = h->plans[j];
    for (int64_t b = 0; b < p.num_full; ++b) bt[(size_t)(p.first_block + b)] = (uint32_t)j;
    bt[(size_t)p.last_block] = (uint32_t)j;
    const TensorDesc d = desc_of(p, h->planes);
    for (TableSlot& t : h->slots) t.h[j] = d;
  }
  hipStream_t s = (hipStream_t)stream;
  if ((e = hipMemcpy(h->d_block_tensor, bt.data(), bt.size() * 4, hipMemcpyHostToDevice)) != hipSuccess) {
    release(h);
    return hip_fail(e, "uploading the block table");
  }
  if ((e = hipMemsetAsync(state, 0, total, s)) != hipSuccess) {
    release(h);
    return hip_fail(e, "clearing the state buffer");
  }
  *out = h;
  clear_error();
  return MICROADAM_OK;
}

int microadam_step(microadam_handle h, void* const* params, const void* const* grads,
                   int32_t n_tensors, double lr, void* stream) {
  int rc = check_handle(h);
  if (rc) return rc;
  if (n_tensors != (int32_t)h->plans.size())
    return fail(MICROADAM_ERR_SHAPE, "n_tensors differs from microadam_init");
  if (!params || !grads) return fail(MICROADAM_ERR_INVALID_ARG, "params / grads is NULL");
  for (int32_t j = 0; j < n_tensors; ++j) {
    if (!params[j] || !grads[j]) return fail(MICROADAM_ERR_INVALID_ARG, "a param or grad pointer is NULL");
    if ((uintptr_t)params[j] % 16 || (uintptr_t)grads[j] % 16)
      return fail(MICROADAM_ERR_INVALID_ARG, "param and grad pointers must be 16-byte aligned");
  }
  if (std::isnan(lr)) lr = h->cfg.lr;
  if (!std::isfinite(lr)) return fail(MICROADAM_ERR_INVALID_ARG, "lr must be finite");
  rc = check_device(h);
  if (rc) return rc;
  hipStream_t s = (hipStream_t)stream;
  hipError_t e;

  // Find a device table holding exactly these addresses, else refill the
  // least recently used one (its staging buffer is rewritten only after its
  // previous upload has been read; the upload is ordered on `s` after every
  // earlier launch on `s`).
  int slot = -1;
  for (int i = 0; i < kTableSlots && slot < 0; ++i) {
    const TableSlot& t = h->slots[i];
    if (!t.last_use) continue;
    bool same = true;
    for (int32_t j = 0; j < n_tensors && same; ++j)
      same = t.h[j].param == params[j] && t.h[j].grad == grads[j];
    if (same) slot = i;
  }
  if (slot < 0) {
    slot = 0;
    for (int i = 1; i < kTableSlots; ++i)
      if (h->slots[i].last_use < h->slots[slot].last_use) slot = i;
    TableSlot& t = h->slots[slot];
    if ((e = hipEventSynchronize(t.upload_done)) != hipSuccess) return hip_fail(e, "hipEventSynchronize");
    for (int32_t j = 0; j < n_tensors; ++j) {
      t.h[j].param = params[j];
      t.h[j].grad = grads[j];
    }
    if ((e = hipMemcpyAsync(t.d, t.h, h->plans.size() * sizeof(TensorDesc), hipMemcpyHostToDevice,
                            s)) != hipSuccess)
      return hip_fail(e, "uploading the tensor table");
    if ((e = hipEventRecord(t.upload_done, s)) != hipSuccess) return hip_fail(e, "hipEventRecord");
  }
  h->slots[slot].last_use = ++h->use_clock;
  h->current = slot;

  const int64_t t = h->t + 1;
  StepParams p;
  fill_constants(h, t, lr, p);
  const bool prof = h->profiling;
  // a profiled step takes the next event set of the ring, first adding the
  // step it held (steps ago, so normally done) to the totals
  const int pslot = prof ? (int)(h->prof_count % microadam_handle_s::kProfSlots) : 0;
  if (prof && (e = fold_slot(h, pslot)) != hipSuccess) return hip_fail(e, "reading the kernel timers");
  auto rec = [&](int i) { return prof ? hipEventRecord(h->ev[pslot][i], s) : hipSuccess; };
  rc = queue_step(p, h->fused, h->planes.big, h->param_bf16, h->grad_bf16, h->value_f32, s, rec);
  if (rc) return rc;
  h->timed = prof;
  if (prof) {
    h->pending[pslot] = true;
    h->prof_slot = pslot;
    ++h->prof_count;
  }
  if ((e = hipEventRecord(h->step_done, s)) != hipSuccess) return hip_fail(e, "hipEventRecord");
  h->t = t;
  return MICROADAM_OK;
}

int microadam_destroy(microadam_handle h) {
  release(h);
  return MICROADAM_OK;
}

int64_t microadam_get_step(microadam_handle h) {
  if (!h) return fail(MICROADAM_ERR_INVALID_ARG, "handle is NULL");
  return h->t;
}

int microadam_set_step(microadam_handle h, int64_t t) {
  int rc = check_handle(h);
  if (rc) return rc;
  if (t < 0) return fail(MICROADAM_ERR_INVALID_ARG, "t must be >= 0");
  h->t = t;
  return MICROADAM_OK;
}

int microadam_tensor_layout(microadam_handle h, int32_t tensor, microadam_layout* out) {
  int rc = check_handle(h);
  if (rc) return rc;
  if (!out) return fail(MICROADAM_ERR_INVALID_ARG, "out is NULL");
  if (tensor < 0 || tensor >= (int32_t)h->plans.size())
    return fail(MICROADAM_ERR_INVALID_ARG, "tensor index out of range");
  const TensorPlan& p = h->plans[(size_t)tensor];
  std::memset(out, 0, sizeof(*out));
  out->numel = p.numel;
  out->num_blocks = p.num_blocks;
  out->num_buckets = p.num_buckets;
  out->k_full = p.k_full;
  out->k_last = p.k_last;
  out->entry_bytes = entry_bytes(&h->cfg);
  out->first_block = p.first_block;
  out->last_block = p.last_block;
  out->ef_plane = h->planes.ef;
  out->ef_stride = h->planes.ef_stride;
  out->stats_plane = h->planes.big ? h->planes.stats + (uint64_t)p.first_bucket * 8 : h->planes.stats;
  out->stats_stride = h->planes.stats_stride;
  out->bucket_table_bytes = h->planes.table_bytes;
  out->window_plane = h->planes.win;
  out->window_stride = h->planes.win_stride;
  return MICROADAM_OK;
}

int microadam_debug_moments(microadam_handle h, int32_t tensor, float* mhat, float* vhat,
                            void* stream) {
  int rc = check_handle(h);
  if (rc) return rc;
  if (tensor < 0 || tensor >= (int32_t)h->plans.size())
    return fail(MICROADAM_ERR_INVALID_ARG, "tensor index out of range");
  if (!mhat || !vhat) return fail(MICROADAM_ERR_INVALID_ARG, "mhat / vhat is NULL");
  if (h->t < 1 || h->current < 0) return fail(MICROADAM_ERR_INVALID_ARG, "no step has been taken");
  rc = check_device(h);
  if (rc) return rc;
  StepParams p;
  fill_constants(h, h->t, h->cfg.lr, p);
  const TensorPlan& tp = h->plans[(size_t)tensor];
  hipError_t e = hipSuccess;
  if (tp.num_full > 0)
    e = microadam::launch_moments(p, tp.first_block, tp.num_full, mhat, vhat, h->value_f32,
                                  (hipStream_t)stream);
  if (e == hipSuccess && tp.num_full < tp.num_blocks)
    e = microadam::launch_moments(p, tp.last_block, 1, mhat, vhat, h->value_f32, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "launching the moment kernel");
  return MICROADAM_OK;
}

int microadam_step_kernels(microadam_handle h) {
  int rc = check_handle(h);
  if (rc) return rc;
  return h->fused ? 1 : h->planes.big ? 4 : h->d_thr ? 4 : 2;
}

int microadam_set_profiling(microadam_handle h, int32_t on) {
  int rc = check_handle(h);
  if (rc) return rc;
  if (on && !h->ev[microadam_handle_s::kProfSlots - 1][3]) {
    rc = check_device(h);
    if (rc) return rc;
    for (auto& set : h->ev)
      for (hipEvent_t& e : set) {
        if (e) continue;
        const hipError_t err = hipEventCreate(&e);
        if (err != hipSuccess) return hip_fail(err, "hipEventCreate");
      }
  }
  if (on) {  // a new total starts; steps not yet added to the old one are dropped
    for (bool& n : h->pending) n = false;
    h->prof_count = 0;
    h->total_ms[0] = h->total_ms[1] = 0.0;
    h->total_steps = 0;
    h->timed = false;
  }
  h->profiling = on != 0;
  return MICROADAM_OK;
}

int microadam_kernel_times(microadam_handle h, float* out_ms) {
  int rc = check_handle(h);
  if (rc) return rc;
  if (!out_ms) return fail(MICROADAM_ERR_INVALID_ARG, "out_ms is NULL");
  if (!h->timed) return fail(MICROADAM_ERR_INVALID_ARG, "the last step was not profiled");
  hipError_t e;
  if ((e = hipEventSynchronize(h->step_done)) != hipSuccess) return hip_fail(e, "hipEventSynchronize");
  if ((e = slot_times(h, h->prof_slot, out_ms)) != hipSuccess) return hip_fail(e, "hipEventElapsedTime");
  return MICROADAM_OK;
}

int microadam_kernel_times_total(microadam_handle h, float* out_ms, int64_t* out_steps) {
  int rc = check_handle(h);
  if (rc) return rc;
  if (!out_ms || !out_steps) return fail(MICROADAM_ERR_INVALID_ARG, "out_ms or out_steps is NULL");
  for (int k = 0; k < microadam_handle_s::kProfSlots; ++k) {
    const hipError_t e = fold_slot(h, k);
    if (e != hipSuccess) return hip_fail(e, "reading the kernel timers");
  }
  out_ms[0] = (float)h->total_ms[0];
  out_ms[1] = (float)h->total_ms[1];
  *out_steps = h->total_steps;
  h->total_ms[0] = h->total_ms[1] = 0.0;
  h->total_steps = 0;
  return MICROADAM_OK;
}

}  // extern "C"

// ------------------------------------------------- the no-allocation step
namespace {
constexpr int32_t kNoAllocMaxTensors = 4096;
constexpr int kNoAllocMaxDevices = 64;
constexpr size_t kNoAllocWeightBytes = 2 * microadam::kMaxWindow * sizeof(float);
constexpr size_t kNoAllocScratchBytes = kNoAllocWeightBytes + (size_t)kNoAllocMaxTensors * sizeof(TensorDesc);

// Host image of the scratch array: the window weights, then the tensor table.
struct NoAllocImage {
  float wpow[2 * microadam::kMaxWindow];
  TensorDesc desc[kNoAllocMaxTensors];
};
static_assert(offsetof(NoAllocImage, desc) == kNoAllocWeightBytes, "weights, then the table");
static_assert(sizeof(NoAllocImage) == kNoAllocScratchBytes, "the image fills the scratch array");

std::mutex g_noalloc_mu;                    // guards the host image and the addresses below
void* g_scratch_dev[kNoAllocMaxDevices];    // per device: the address of its `scratch`
TensorPlan g_noalloc_plans[kNoAllocMaxTensors];
NoAllocImage g_noalloc_image;
}  // namespace

// Device memory of microadam_step_noalloc (the window weights and the tensor
// table of the last call), one copy per GPU for the life of the process.  In
// host code the name only stands for the symbol: its device address comes
// from hipGetSymbolAddress, once per device.
static __device__ __align__(256) uint8_t scratch[kNoAllocScratchBytes];

extern "C" {

int microadam_step_noalloc(const microadam_config* cfg, const int64_t* numels, int32_t n_tensors,
                           int32_t param_dtype, int32_t grad_dtype, void* state, uint64_t state_bytes,
                           int64_t t, void* const* params, const void* const* grads, double lr, void* stream) {
  int rc = validate_config(cfg);
  if (rc) return rc;
  if (n_tensors < 1) return fail(MICROADAM_ERR_INVALID_ARG, "n_tensors must be >= 1");
  if (n_tensors > kNoAllocMaxTensors)
    return fail(MICROADAM_ERR_UNSUPPORTED, "microadam_step_noalloc takes at most 4096 tensors");
  if ((param_dtype != MICROADAM_F32 && param_dtype != MICROADAM_BF16) ||
      (grad_dtype != MICROADAM_F32 && grad_dtype != MICROADAM_BF16))
    return fail(MICROADAM_ERR_INVALID_ARG, "param_dtype / grad_dtype must be F32 or BF16");
  if (t < 1) return fail(MICROADAM_ERR_INVALID_ARG, "t must be >= 1");
  if (!state) return fail(MICROADAM_ERR_INVALID_ARG, "state is NULL");
  if ((uintptr_t)state % kAlign) return fail(MICROADAM_ERR_INVALID_ARG, "state must be 256-byte aligned");
  if (!params || !grads) return fail(MICROADAM_ERR_INVALID_ARG, "params / grads is NULL");
  for (int32_t j = 0; j < n_tensors; ++j) {
    if (!params[j] || !grads[j]) return fail(MICROADAM_ERR_INVALID_ARG, "a param or grad pointer is NULL");
    if ((uintptr_t)params[j] % 16 || (uintptr_t)grads[j] % 16)
      return fail(MICROADAM_ERR_INVALID_ARG, "param and grad pointers must be 16-byte aligned");
  }
  if (std::isnan(lr)) lr = cfg->lr;
  if (!std::isfinite(lr)) return fail(MICROADAM_ERR_INVALID_ARG, "lr must be finite");

  std::lock_guard<std::mutex> lock(g_noalloc_mu);
  Planes pl;
  rc = make_plan(cfg, numels, n_tensors, g_noalloc_plans, pl);
  if (rc) return rc;
  if (state_bytes < pl.total) return fail(MICROADAM_ERR_STATE_SIZE, "state buffer smaller than microadam_state_bytes");
  rc = check_launch_size(cfg, pl);
  if (rc) return rc;
  const int32_t k_full = g_noalloc_plans[0].k_full;
  const int32_t value_f32 = cfg->window_value_dtype == MICROADAM_F32;
  if (microadam::step_lds_bytes(cfg->topk_block, k_full, value_f32) > kMaxLds)
    return fail(MICROADAM_ERR_UNSUPPORTED, "k per block too large for the LDS budget");
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kNoAllocMaxDevices) return fail(MICROADAM_ERR_UNSUPPORTED, "device number above 63");
  if (!g_scratch_dev[dev]) {
    // first call on this device (current): where its copy of `scratch` lives
    void* ptr = nullptr;
    if ((e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch))) != hipSuccess)
      return hip_fail(e, "hipGetSymbolAddress");
    if (!ptr) return fail(MICROADAM_ERR_HIP, "hipGetSymbolAddress returned NULL");
    g_scratch_dev[dev] = ptr;
  }
  uint8_t* const dev_scratch = (uint8_t*)g_scratch_dev[dev];
  window_weights(cfg, g_noalloc_image.wpow);
  for (int32_t j = 0; j < n_tensors; ++j) {
    TensorDesc d = desc_of(g_noalloc_plans[j], pl);
    d.param = params[j];
    d.grad = grads[j];
    g_noalloc_image.desc[j] = d;
  }
  hipStream_t s = (hipStream_t)stream;
  // the weights and this call's part of the table; the copy is ordered after
  // earlier work on `s`, and the host image is not needed once the call
  // returns (a copy from pageable host memory has read it by then)
  if ((e = hipMemcpyAsync(dev_scratch, &g_noalloc_image, kNoAllocWeightBytes + (size_t)n_tensors * sizeof(TensorDesc),
                          hipMemcpyHostToDevice, s)) != hipSuccess)
    return hip_fail(e, "uploading the tensor table");
  const int32_t param_bf16 = param_dtype == MICROADAM_BF16, grad_bf16 = grad_dtype == MICROADAM_BF16;
  StepParams p;
  // no block table: the kernels find a block's tensor by binary search
  fill_step_params(*cfg, pl, k_full, n_tensors, bucket_log2_of(cfg, pl), t, lr,
                   (const TensorDesc*)(dev_scratch + kNoAllocWeightBytes), nullptr, (const float*)dev_scratch,
                   (uint8_t*)state, p);
  const bool fused = use_fused(cfg, pl, k_full, param_bf16, grad_bf16);
  rc = queue_step(p, fused, pl.big, param_bf16, grad_bf16, value_f32, s, [](int) { return hipSuccess; });
  if (rc) return rc;
  clear_error();
  return MICROADAM_OK;
}

const char* microadam_error_string(int code) {
  switch (code) {
    case MICROADAM_OK: return "ok";
    case MICROADAM_ERR_INVALID_ARG: return "invalid argument";
    case MICROADAM_ERR_UNSUPPORTED: return "unsupported configuration";
    case MICROADAM_ERR_SHAPE: return "tensor list differs from init";
    case MICROADAM_ERR_STATE_SIZE: return "state buffer too small";
    case MICROADAM_ERR_HIP: return "HIP runtime error";
    case MICROADAM_ERR_NO_MEMORY: return "out of memory";
    default: return "unknown error code";
  }
}

const char* microadam_last_error(void) { return g_last_error; }

}  // extern "C"
