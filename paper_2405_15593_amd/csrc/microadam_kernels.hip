// MicroAdam step kernels for CDNA4 (gfx950).
//
// One optimizer step is two launches over all Top-K blocks (B_d elements of
// one tensor each; blocks share nothing):
//
//   select_kernel   one workgroup per block:
//     1. a = g + Q^-1(e)                          (Algorithm 1; Algorithm 2, Q^-1)
//     2. block Top-K of |a|, lower index wins ties (Section 3.1, "Top-K")
//     3. the new window row (I, bf16(V)) is stored (Section 3.2)
//     4. a[I] = 0; bucket (delta, Delta) = (min, max) by lane shuffles;
//        e = Q(a, delta, Delta), two 4-bit codes per byte (Algorithm 1; Section 3.1)
//
//   update_kernel   one workgroup per block:
//     5. one wave rebuilds m-hat, v-hat of the block's window entries in LDS
//        from the m rows with weights beta^(t-s) (Algorithm 2, AdamStats)
//     6. every wave applies theta <- (1 - eta*lambda) theta
//        - eta m / (eps + sqrt(v)) to its elements (Algorithm 1; Algorithm 4)
//
// Splitting the step costs one extra read of the new window row (4 bytes per
// kept entry) and lets each kernel keep a small register and LDS footprint.
//
// Element layout inside a block: thread `tid` owns the 16 consecutive
// elements tid*16 + [0, 16), handled as two vectors of 8.  An EF bucket of
// B_q >= 16 elements is held by B_q/16 neighbouring lanes; with B_q = 8 each
// vector is one bucket.
//
// Arithmetic that decides an integer (EF decode, accumulator, Top-K order,
// bucket min/max, codes) is binary32 with one rounding per written operation
// (the file is compiled with -ffp-contract=off); the only fused operations in
// that part are in div15, which is exact, and the code brackets of step 4,
// which are checked against the exact quotient's rounding.  The device code
// is compiled without IEEE NaN handling (min/max do not quiet NaNs):
// gradients are taken to be finite.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "microadam_device.h"

namespace microadam {
namespace {

constexpr int kWave = 64;
constexpr int kLaneElems = 16;       // consecutive elements per thread
constexpr int kRegion = 32;          // candidate vectors one wave can hand to the leader
constexpr int kCand = 256;           // candidate elements the leader resolves
constexpr uint32_t kNoEntry = 0xFFFFFFFFu;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __amdgpu_buffer_rsrc_t Rsrc;

// ---------------------------------------------------------------- wave ops
__device__ __forceinline__ uint64_t ballot(bool p) { return __ballot(p); }
__device__ __forceinline__ uint32_t lanes_below(uint64_t m) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}
__device__ __forceinline__ uint32_t popc(uint64_t m) { return (uint32_t)__popcll(m); }
__device__ __forceinline__ uint32_t sgpr(uint32_t x) { return __builtin_amdgcn_readfirstlane(x); }
// A uniform value the compiler must treat as unknown at this point, so that
// tests on it stay where they are written instead of being computed early
// and kept in scalar registers.
__device__ __forceinline__ int opaque(int x) {
  asm volatile("" : "+s"(x));
  return x;
}
// Work-item and workgroup ids straight from the hardware registers (the
// library wrappers behind threadIdx / blockIdx are not inlined into code
// built without IEEE mode).
__device__ __forceinline__ int thread_id() { return (int)__builtin_amdgcn_workitem_id_x(); }
__device__ __forceinline__ int64_t block_id() { return (int64_t)__builtin_amdgcn_workgroup_id_x(); }

template <int CTRL>
__device__ __forceinline__ float dpp_mov(float x) {
  return __builtin_bit_cast(
      float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xF, 0xF, false));
}

// min / max over aligned groups of 2^g neighbouring lanes, g in [0, 5]
// (quad permutes, then half-row and row mirrors, then a lane shuffle).
__device__ __forceinline__ void group_minmax(float& mn, float& mx, int g) {
  if (g >= 1) { mn = __builtin_fminf(mn, dpp_mov<0xB1>(mn)); mx = __builtin_fmaxf(mx, dpp_mov<0xB1>(mx)); }
  if (g >= 2) { mn = __builtin_fminf(mn, dpp_mov<0x4E>(mn)); mx = __builtin_fmaxf(mx, dpp_mov<0x4E>(mx)); }
  if (g >= 3) { mn = __builtin_fminf(mn, dpp_mov<0x141>(mn)); mx = __builtin_fmaxf(mx, dpp_mov<0x141>(mx)); }
  if (g >= 4) { mn = __builtin_fminf(mn, dpp_mov<0x140>(mn)); mx = __builtin_fmaxf(mx, dpp_mov<0x140>(mx)); }
  if (g >= 5) {
    mn = __builtin_fminf(mn, __shfl_xor(mn, 16, kWave));
    mx = __builtin_fmaxf(mx, __shfl_xor(mx, 16, kWave));
  }
}

// d / 15 correctly rounded for every finite d >= +0: q0 = d * fl(1/15), then
// one FMA residual step (checked exhaustively against IEEE division).
__device__ __forceinline__ float div15(float d) {
  const float r = 1.0f / 15.0f;
  const float q0 = d * r;
  const float e = __builtin_fmaf(-q0, 15.0f, d);
  return __builtin_fmaf(e, r, q0);
}

// Byte n of x as a float (v_cvt_f32_ubyte{n}); the compiler does not form
// these from shifts and masks of packed nibbles.
template <int N>
__device__ __forceinline__ float ubyte(uint32_t x) {
  float r;
  if constexpr (N == 0) asm("v_cvt_f32_ubyte0 %0, %1" : "=v"(r) : "v"(x));
  else if constexpr (N == 1) asm("v_cvt_f32_ubyte1 %0, %1" : "=v"(r) : "v"(x));
  else if constexpr (N == 2) asm("v_cvt_f32_ubyte2 %0, %1" : "=v"(r) : "v"(x));
  else asm("v_cvt_f32_ubyte3 %0, %1" : "=v"(r) : "v"(x));
  return r;
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }
__device__ __forceinline__ uint32_t to_bf16_bits(float x) {
  const __bf16 b = (__bf16)x;  // v_cvt_pk_bf16_f32: round half to even
  return (uint32_t)__builtin_bit_cast(uint16_t, b);
}

// Buffer resource over [base, base + bytes): loads past the end read 0 and
// stores past it are dropped.  Base and size are workgroup-uniform; reading
// them through readfirstlane keeps the resource in scalar registers.
__device__ __forceinline__ Rsrc make_rsrc(const void* base, uint32_t bytes) {
  const uint64_t a = (uint64_t)base;
  const uint64_t u = ((uint64_t)sgpr((uint32_t)(a >> 32)) << 32) | sgpr((uint32_t)a);
  return __builtin_amdgcn_make_buffer_rsrc((void*)u, (short)0, sgpr(bytes), 0x00020000);
}

// Tables the kernel only reads, addressed as constant memory so that their
// uniform loads become scalar loads.
template <typename T>
__device__ __forceinline__ const __attribute__((address_space(4))) T* constant_ptr(const T* p) {
  return (const __attribute__((address_space(4))) T*)p;
}

__device__ __forceinline__ TensorDesc load_desc(const __attribute__((address_space(4))) TensorDesc* d) {
  TensorDesc r;
  r.param = d->param;
  r.grad = d->grad;
  r.numel = d->numel;
  r.first_block = d->first_block;
  r.num_blocks = d->num_blocks;
  r.last_block = d->last_block;
  r.k_full = d->k_full;
  r.k_last = d->k_last;
  r.s_last = d->s_last;
  r.num_full = d->num_full;
  return r;
}

__device__ __forceinline__ uint32_t key_of(float a) { return __float_as_uint(a) & 0x7FFFFFFFu; }

// Workgroup barrier that orders LDS only.  The waves of a workgroup exchange
// data through LDS alone, so no wait for outstanding global loads or stores
// is needed here.
__device__ __forceinline__ void lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// -------------------------------------------------------- element vectors
// Raw storage of 8 consecutive elements of a bf16 or float32 tensor.
template <bool BF16> struct Raw8 { u32x4 w[BF16 ? 1 : 2]; };

// The resource of a block covers its elements rounded up to whole 16-byte
// chunks.  A 16-byte-aligned chunk holding a valid element lies inside the
// tensor's allocation page, and chunks past the rounded end read 0, so the
// 16-byte loads never touch memory outside that page; the few elements past
// the end of a ragged tensor are masked to 0 by the caller.
template <bool BF16>
__device__ __forceinline__ Raw8<BF16> load8(Rsrc r, uint32_t elem) {
  Raw8<BF16> x;
  constexpr uint32_t es = BF16 ? 2 : 4;
  x.w[0] = __builtin_amdgcn_raw_buffer_load_b128(r, elem * es, 0, 0);
  if constexpr (!BF16) x.w[1] = __builtin_amdgcn_raw_buffer_load_b128(r, elem * es + 16, 0, 0);
  return x;
}

template <bool BF16>
__device__ __forceinline__ uint32_t vec_bytes(int s) {
  return ((uint32_t)s * (BF16 ? 2u : 4u) + 15u) & ~15u;
}

template <bool BF16>
__device__ __forceinline__ void unpack8(const Raw8<BF16>& x, float out[8]) {
  if constexpr (BF16) {
#pragma unroll
    for (int h = 0; h < 4; ++h) { out[2 * h] = bf16_lo(x.w[0][h]); out[2 * h + 1] = bf16_hi(x.w[0][h]); }
  } else {
#pragma unroll
    for (int h = 0; h < 4; ++h) { out[h] = __uint_as_float(x.w[0][h]); out[4 + h] = __uint_as_float(x.w[1][h]); }
  }
}

// Stores 8 elements; `full` (workgroup-uniform) selects whole-vector stores,
// otherwise only elements below s are written.
template <bool BF16>
__device__ __forceinline__ void store8(Rsrc r, uint32_t elem, int s, bool full, const float in[8]) {
  constexpr uint32_t es = BF16 ? 2 : 4;
  if (full) {
    if constexpr (BF16) {
      u32x4 w;
#pragma unroll
      for (int h = 0; h < 4; ++h) w[h] = to_bf16_bits(in[2 * h]) | (to_bf16_bits(in[2 * h + 1]) << 16);
      __builtin_amdgcn_raw_buffer_store_b128(w, r, elem * es, 0, 0);
    } else {
      __builtin_amdgcn_raw_buffer_store_b128(u32x4{__float_as_uint(in[0]), __float_as_uint(in[1]),
                                                   __float_as_uint(in[2]), __float_as_uint(in[3])},
                                             r, elem * es, 0, 0);
      __builtin_amdgcn_raw_buffer_store_b128(u32x4{__float_as_uint(in[4]), __float_as_uint(in[5]),
                                                   __float_as_uint(in[6]), __float_as_uint(in[7])},
                                             r, elem * es + 16, 0, 0);
    }
  } else {
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      if ((int)elem + e < s) {
        if constexpr (BF16) __builtin_amdgcn_raw_buffer_store_b16((uint16_t)to_bf16_bits(in[e]), r, (elem + e) * 2, 0, 0);
        else __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(in[e]), r, (elem + e) * 4, 0, 0);
      }
    }
  }
}

// ------------------------------------------------------- window entries
// bf16 values: one word (index | bf16 << 16); f32 values: (index, value).
template <bool VF32> struct Entry {
  typedef typename std::conditional<VF32, u32x2, uint32_t>::type T;
  __device__ static T make(uint32_t idx, float v) {
    if constexpr (VF32) return u32x2{idx, __float_as_uint(v)};
    else return idx | (to_bf16_bits(v) << 16);
  }
  __device__ static T none() {
    if constexpr (VF32) return u32x2{kNoEntry, 0u};
    else return kNoEntry;
  }
  __device__ static uint32_t idx(T e) {
    if constexpr (VF32) return e[0];
    else return e == kNoEntry ? kNoEntry : (e & 0xFFFFu);
  }
  __device__ static float val(T e) {
    if constexpr (VF32) return __uint_as_float(e[1]);
    else return __uint_as_float(e & 0xFFFF0000u);
  }
  __device__ static T load(Rsrc r, uint32_t entry) {
    if constexpr (VF32) return __builtin_amdgcn_raw_buffer_load_b64(r, entry * 8, 0, 0);
    else return __builtin_amdgcn_raw_buffer_load_b32(r, entry * 4, 0, 0);
  }
  __device__ static void store(Rsrc r, uint32_t entry, T e) {
    if constexpr (VF32) __builtin_amdgcn_raw_buffer_store_b64(e, r, entry * 8, 0, 0);
    else __builtin_amdgcn_raw_buffer_store_b32(e, r, entry * 4, 0, 0);
  }
};

// ------------------------------------------------------- block geometry
// Everything a workgroup needs to know about its block (workgroup-uniform).
struct Block {
  int64_t e0;             // first element of the block in its tensor
  TensorDesc desc;
  int s;                  // valid elements
  int kq;                 // window entries per row
};

__device__ __forceinline__ Block locate(const StepParams& p, int64_t gb) {
  Block b;
  const uint32_t j = constant_ptr(p.block_tensor)[gb];
  b.desc = load_desc(constant_ptr(p.tensors) + j);
  const bool last = (int32_t)gb == (int32_t)b.desc.last_block;
  const int32_t q = last ? (int32_t)b.desc.num_blocks - 1 : (int32_t)(gb - b.desc.first_block);
  b.e0 = (int64_t)q * p.block;
  b.s = last ? b.desc.s_last : p.block;
  b.kq = last ? b.desc.k_last : b.desc.k_full;
  return b;
}

// Geometry of one block as the update kernel carries it.
struct Span {
  uint64_t base;          // byte address of the block's first parameter
  int64_t e0;             // first element of the block in its tensor
  int32_t gb;             // global block number
  int32_t s;              // valid elements
  int32_t kq;             // window entries per row
};

// The tensor of the full blocks a workgroup walks through in order; the
// tables are read again only when the walk crosses into another tensor.
// Global block numbers are below 2^31 (checked at init) and are compared as
// 32-bit values, which keeps the comparisons scalar.
struct Cursor {
  uint64_t param;
  int32_t first;          // first global block of the tensor
  int32_t end;            // first global block past its full blocks (0: none yet)
};

// Full block gb (gb < n_full): B_d elements, k_full entries per row.
__device__ __forceinline__ Span seek_full(const StepParams& p, Cursor& c, int32_t gb, uint32_t elem_bytes) {
  if (gb >= c.end) {
    const uint32_t j = constant_ptr(p.block_tensor)[gb];
    const __attribute__((address_space(4))) TensorDesc* d = constant_ptr(p.tensors) + j;
    c.param = (uint64_t)d->param;
    c.first = (int32_t)d->first_block;
    c.end = c.first + d->num_full;
  }
  Span u;
  u.gb = gb;
  u.e0 = (int64_t)(gb - c.first) * p.block;
  u.base = c.param + (uint64_t)u.e0 * elem_bytes;
  u.s = p.block;
  u.kq = p.k_full;
  return u;
}

// Any block: full, or the ragged last block of its tensor.
__device__ __forceinline__ Span span_of(const StepParams& p, int32_t gb, uint32_t elem_bytes) {
  const Block b = locate(p, gb);
  Span u;
  u.gb = gb;
  u.e0 = b.e0;
  u.base = (uint64_t)b.desc.param + (uint64_t)b.e0 * elem_bytes;
  u.s = b.s;
  u.kq = b.kq;
  return u;
}

template <int EW>
__device__ __forceinline__ Rsrc window_rsrc(const StepParams& p, int64_t gb, int kq) {
  const uint64_t slot_bytes = (uint64_t)p.window * p.k_full * EW * 4;
  return make_rsrc(p.state + p.win_plane + (uint64_t)gb * slot_bytes, (uint32_t)(p.window * kq * EW * 4));
}

// ------------------------------------------------------- select LDS
template <int NT>
struct SelectLds {
  static constexpr int NW = NT / kWave;
  float* regv;        // [NW][kRegion][8] candidate vectors per wave
  uint32_t* regi;     // [NW][kRegion] their first element index
  float* cval;        // candidate values (first half of regv, once read)
  uint32_t* cidx;     // candidate indices (second half of regv, once read)
  uint32_t* misc;     // 64 words: counts, wave bounds, broadcast, reductions
  __device__ explicit SelectLds(uint32_t* smem) {
    regv = (float*)smem;
    regi = (uint32_t*)(regv + NW * kRegion * 8);
    cval = regv;
    cidx = (uint32_t*)(regv + NW * kRegion * 4);
    misc = regi + NW * kRegion;
  }
  static constexpr size_t words() { return (size_t)NW * kRegion * 9 + 64; }
};
// misc word offsets
enum { M_COUNT = 0 /* [NW] */, M_WL = 8 /* [NW] */, M_GEN = 12, M_T = 13, M_ILAST = 14,
       M_NOTIE = 15, M_RED0 = 16, M_RED1 = 32, M_RED2 = 48 /* 16 words each */ };

// Exclusive prefix, in element order, of per-(thread, vector) counts <= 8.
// base[v] = counted elements before this thread's vector v.  One barrier;
// `red` (NW words) must not be reused until a later barrier.
template <int NT>
__device__ __forceinline__ void wg_scan(const uint32_t (&cnt)[2], uint32_t (&base)[2], uint32_t* red) {
  constexpr int NW = NT / kWave;
  const int lane = thread_id() & (kWave - 1), wave = (int)sgpr(thread_id() / kWave);
  const uint32_t c = cnt[0] + cnt[1];  // <= 16
  uint32_t pre = 0, tot = 0;
#pragma unroll
  for (int b = 0; b < 5; ++b) {
    const uint64_t m = ballot((c >> b) & 1u);
    pre += lanes_below(m) << b;
    tot += popc(m) << b;
  }
  if (lane == 0) red[wave] = tot;
  lds_sync();
  uint32_t run = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) run += (w < wave) ? red[w] : 0u;
  base[0] = run + pre;
  base[1] = base[0] + cnt[0];
}

// Workgroup-wide count of elements flagged in two 8-bit masks.  One barrier;
// consecutive calls must use different `red` buffers (NW words).
template <int NT>
__device__ __forceinline__ uint32_t wg_count(const uint32_t (&mask)[2], uint32_t* red) {
  constexpr int NW = NT / kWave;
  const int lane = thread_id() & (kWave - 1), wave = (int)sgpr(thread_id() / kWave);
  const uint32_t c = __popc(mask[0]) + __popc(mask[1]);  // <= 16
  uint32_t tot = 0;
#pragma unroll
  for (int b = 0; b < 5; ++b) tot += popc(ballot((c >> b) & 1u)) << b;
  if (lane == 0) red[wave] = tot;
  lds_sync();
  uint32_t s = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) s += red[w];
  return s;
}

// ============================================================ select
template <int NT, bool GBF16, bool VF32>
__global__ void __launch_bounds__(NT) select_kernel(StepParams p) {
  constexpr int NW = NT / kWave;
  constexpr int CAP = NT * kLaneElems;
  constexpr int EW = VF32 ? 2 : 1;
  constexpr uint32_t kCandCap = (uint32_t)(kCand < NW * kRegion * 4 ? kCand : NW * kRegion * 4);
  using E = Entry<VF32>;
  extern __shared__ __align__(16) uint32_t smem[];
  const SelectLds<NT> l(smem);

  const int tid = thread_id(), lane = tid & (kWave - 1), wave = (int)sgpr(tid / kWave);
  const uint32_t eb = (uint32_t)tid * kLaneElems;  // first element of this thread
  const int bl = p.bucket_log2;
  const bool pair_buckets = bl == 3;               // B_q = 8: one bucket per vector
  const int64_t gb = block_id();

  // The block's EF codes and bucket pairs are addressed by gb alone, so their
  // loads go out before the tensor lookup that the gradient needs.
  const uint32_t nbk = (uint32_t)(p.block >> bl);
  const Rsrc re = make_rsrc(p.state + p.ef_plane + (uint64_t)gb * (p.block >> 1), (uint32_t)(p.block >> 1));
  const Rsrc rs = make_rsrc(p.state + p.stats_plane + (uint64_t)gb * nbk * 8, nbk * 8);
  u32x4 st;
  if (pair_buckets) {
    st = __builtin_amdgcn_raw_buffer_load_b128(rs, eb, 0, 0);
  } else {
    const u32x2 t = __builtin_amdgcn_raw_buffer_load_b64(rs, (eb >> bl) * 8, 0, 0);
    st = u32x4{t[0], t[1], 0u, 0u};
  }
  const u32x2 codes = __builtin_amdgcn_raw_buffer_load_b64(re, eb >> 1, 0, 0);
  const Block b = locate(p, gb);
  const int s = b.s, kq = b.kq;
  const bool full = s == CAP;
  const Rsrc rg = make_rsrc((const uint8_t*)b.desc.grad + b.e0 * (GBF16 ? 2 : 4), vec_bytes<GBF16>(s));
  Raw8<GBF16> graw[2];
#pragma unroll
  for (int v = 0; v < 2; ++v) graw[v] = load8<GBF16>(rg, eb + v * 8);

  // ---------------------------------------------- 1. a = g + Q^-1(e)
  float a[2][8];
  {
    const float lo0 = __uint_as_float(st[0]), hi0 = __uint_as_float(st[1]);
    const float u0 = div15(hi0 - lo0);
    const float lo1 = pair_buckets ? __uint_as_float(st[2]) : lo0;
    const float u1 = pair_buckets ? div15(__uint_as_float(st[3]) - lo1) : u0;
#pragma unroll
    for (int v = 0; v < 2; ++v) {
      const float lo = v ? lo1 : lo0, u = v ? u1 : u0;
      const uint32_t w = codes[v];
      const uint32_t ev = w & 0x0F0F0F0Fu, od = (w >> 4) & 0x0F0F0F0Fu;
      float g[8], c[8];
      unpack8<GBF16>(graw[v], g);
      c[0] = ubyte<0>(ev); c[2] = ubyte<1>(ev); c[4] = ubyte<2>(ev); c[6] = ubyte<3>(ev);
      c[1] = ubyte<0>(od); c[3] = ubyte<1>(od); c[5] = ubyte<2>(od); c[7] = ubyte<3>(od);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float sc = c[e] * u;
        const float d = sc + lo;
        a[v][e] = g[e] + d;
      }
    }
  }
  // elements of this thread below the end of the block: [0, rem)
  const int rem = s - (int)eb;
  if (!full) {  // elements past the end of the tensor are 0 and never kept
#pragma unroll
    for (int v = 0; v < 2; ++v)
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (v * 8 + e >= rem) a[v][e] = 0.0f;
  }

  // ---------------------------------------------- 2. Top-K threshold
  // Lower bound L: per wave, the ceil(k/NW)-th largest lane maximum of |a|
  // (resolved on its top 13 bits); at least k elements are >= the minimum
  // over waves.
  float vmax[2];
#pragma unroll
  for (int v = 0; v < 2; ++v) {
    const float m0 = __builtin_fmaxf(__builtin_fmaxf(__builtin_fabsf(a[v][0]), __builtin_fabsf(a[v][1])), __builtin_fabsf(a[v][2]));
    const float m1 = __builtin_fmaxf(__builtin_fmaxf(__builtin_fabsf(a[v][3]), __builtin_fabsf(a[v][4])), __builtin_fabsf(a[v][5]));
    const float m2 = __builtin_fmaxf(__builtin_fmaxf(m0, m1), __builtin_fabsf(a[v][6]));
    vmax[v] = __builtin_fmaxf(m2, __builtin_fabsf(a[v][7]));
  }
  const bool fast_k = kq <= kWave * NW;
  {
    const uint32_t lmax = __float_as_uint(__builtin_fmaxf(vmax[0], vmax[1]));
    const int kw = (kq + NW - 1) / NW;
    uint32_t P = 0;
#pragma unroll
    for (int bit = 30; bit >= 18; --bit) {
      const uint32_t c = P | (1u << bit);
      if ((int)popc(ballot(lmax >= c)) >= kw) P = c;
    }
    if (lane == 0) l.misc[M_WL + wave] = P;
  }
  lds_sync();  // B1 ------------------------------------------------

  // The leader wave resolves the threshold; it rotates with the block so that
  // the leaders of the workgroups sharing a compute unit spread over its SIMDs.
  const int leader = (int)(gb & (NW - 1));
  const Rsrc rw = window_rsrc<EW>(p, gb, kq);
  float L;
  {
    uint32_t Lb = l.misc[M_WL];
#pragma unroll
    for (int w = 1; w < NW; ++w) Lb = min(Lb, l.misc[M_WL + w]);
    L = __uint_as_float(sgpr(Lb));
  }
  // candidate vectors, those holding some |a| >= L, handed to the leader in
  // element order (wave, lane, vector)
  {
    const bool f0 = vmax[0] >= L, f1 = vmax[1] >= L;
    const uint64_t m0 = ballot(f0), m1 = ballot(f1);
    const uint32_t pos0 = lanes_below(m0) + lanes_below(m1);
    const uint32_t pos1 = pos0 + (f0 ? 1u : 0u);
    float* rv = l.regv + wave * kRegion * 8;
    uint32_t* ri = l.regi + wave * kRegion;
    if (f0 && pos0 < (uint32_t)kRegion) {
      *(float4*)(rv + pos0 * 8) = make_float4(a[0][0], a[0][1], a[0][2], a[0][3]);
      *(float4*)(rv + pos0 * 8 + 4) = make_float4(a[0][4], a[0][5], a[0][6], a[0][7]);
      ri[pos0] = eb;
    }
    if (f1 && pos1 < (uint32_t)kRegion) {
      *(float4*)(rv + pos1 * 8) = make_float4(a[1][0], a[1][1], a[1][2], a[1][3]);
      *(float4*)(rv + pos1 * 8 + 4) = make_float4(a[1][4], a[1][5], a[1][6], a[1][7]);
      ri[pos1] = eb + 8;
    }
    if (lane == 0) l.misc[M_COUNT + wave] = popc(m0) + popc(m1);
  }
  lds_sync();  // B2 ------------------------------------------------

  bool general;
  {
    uint32_t nvec = 0;
    bool overflow = false;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const uint32_t c = sgpr(l.misc[M_COUNT + w]);
      nvec += c;
      overflow |= c > (uint32_t)kRegion;
    }
    general = !fast_k || L == 0.0f || overflow || nvec > 2u * kWave;
  }
  if (!general && wave == leader) {
    // this lane takes candidate vectors lane and lane + 64 (element order)
    uint32_t src[2];
    bool have[2];
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      const uint32_t j = lane + kWave * r;
      uint32_t off = 0, at = 0;
      bool found = false;
#pragma unroll
      for (int w = 0; w < NW; ++w) {
        const uint32_t cw = sgpr(l.misc[M_COUNT + w]);
        if (!found && j < off + cw) { found = true; at = w * kRegion + (j - off); }
        off += cw;
      }
      have[r] = found;
      src[r] = at;
    }
    // elements with |a| >= L of both vectors, in element order
    float cv[2][8];
    uint32_t base[2], total = 0;
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      const float4 x0 = *(const float4*)(l.regv + src[r] * 8);
      const float4 x1 = *(const float4*)(l.regv + src[r] * 8 + 4);
      cv[r][0] = x0.x; cv[r][1] = x0.y; cv[r][2] = x0.z; cv[r][3] = x0.w;
      cv[r][4] = x1.x; cv[r][5] = x1.y; cv[r][6] = x1.z; cv[r][7] = x1.w;
      uint32_t c = 0;
#pragma unroll
      for (int e = 0; e < 8; ++e) c += (have[r] && __builtin_fabsf(cv[r][e]) >= L) ? 1u : 0u;
      const uint64_t b0 = ballot(c & 1u), b1 = ballot(c & 2u), b2 = ballot(c & 4u), b3 = ballot(c & 8u);
      base[r] = total + lanes_below(b0) + 2u * lanes_below(b1) + 4u * lanes_below(b2) + 8u * lanes_below(b3);
      total += popc(b0) + 2u * popc(b1) + 4u * popc(b2) + 8u * popc(b3);
    }
    const uint32_t cb0 = l.regi[src[0]], cb1 = l.regi[src[1]];
    const uint32_t C = total;
    if (C > kCandCap || C < (uint32_t)kq) {
      if (lane == 0) l.misc[M_GEN] = 1;
    } else {
      // every region read above has returned before the candidate arrays,
      // which reuse the region memory, are written
      __builtin_amdgcn_s_waitcnt(0xC07F);
#pragma unroll
      for (int r = 0; r < 2; ++r) {
        uint32_t pos = base[r];
        const uint32_t cb = r ? cb1 : cb0;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          if (have[r] && __builtin_fabsf(cv[r][e]) >= L) {
            l.cval[pos] = cv[r][e];
            l.cidx[pos] = cb + e;
            ++pos;
          }
        }
      }
      // k-th largest key among the candidates, one bit at a time from the top
      uint32_t ck[4], ci[4];
      float cf[4];
      bool ok[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const uint32_t j = lane + kWave * r;
        ok[r] = j < C;
        cf[r] = ok[r] ? l.cval[j] : 0.0f;
        ci[r] = ok[r] ? l.cidx[j] : 0u;
        ck[r] = ok[r] ? key_of(cf[r]) : 0u;
      }
      const uint32_t nslot = (C + kWave - 1) / kWave;
      uint32_t T = 0;
      if (nslot == 1) {
#pragma unroll
        for (int bit = 30; bit >= 0; --bit) {
          const uint32_t c = T | (1u << bit);
          if (popc(ballot(ck[0] >= c)) >= (uint32_t)kq) T = c;
        }
      } else if (nslot == 2) {
#pragma unroll
        for (int bit = 30; bit >= 0; --bit) {
          const uint32_t c = T | (1u << bit);
          if (popc(ballot(ck[0] >= c)) + popc(ballot(ck[1] >= c)) >= (uint32_t)kq) T = c;
        }
      } else {
        for (int bit = 30; bit >= 0; --bit) {
          const uint32_t c = T | (1u << bit);
          uint32_t n = popc(ballot(ck[0] >= c)) + popc(ballot(ck[1] >= c)) + popc(ballot(ck[2] >= c));
          if (nslot > 3) n += popc(ballot(ck[3] >= c));
          if (n >= (uint32_t)kq) T = c;
        }
      }
      uint32_t ngt = 0, neq = 0;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        ngt += popc(ballot(ok[r] && ck[r] > T));
        neq += popc(ballot(ok[r] && ck[r] == T));
      }
      const uint32_t need = (uint32_t)kq - ngt;  // >= 1 of the keys equal to T are kept
      uint32_t eq_before = 0, sel_before = 0;
      const uint32_t row0 = (uint32_t)p.new_slot * kq;
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const bool gt = ok[r] && ck[r] > T;
        const bool eq = ok[r] && ck[r] == T;
        const uint64_t em = ballot(eq);
        const uint32_t rank = eq_before + lanes_below(em);
        eq_before += popc(em);
        if (eq && rank == need - 1) l.misc[M_ILAST] = ci[r];
        const bool sel = gt || (eq && rank < need);
        const uint64_t sm = ballot(sel);
        const uint32_t pos = sel_before + lanes_below(sm);
        sel_before += popc(sm);
        if (sel) E::store(rw, row0 + pos, E::make(ci[r], cf[r]));
      }
      if (lane == 0) {
        l.misc[M_T] = T;
        l.misc[M_NOTIE] = (neq == need) ? 1u : 0u;
        l.misc[M_GEN] = 0;
      }
    }
  }
  if (!general) {
    lds_sync();  // B3 ----------------------------------------------
    general = sgpr(l.misc[M_GEN]) != 0;
  }

  uint32_t T, i_last;
  bool notie;
  if (!general) {
    T = sgpr(l.misc[M_T]);
    i_last = sgpr(l.misc[M_ILAST]);
    notie = sgpr(l.misc[M_NOTIE]) != 0;
  } else {
    // Exact bitwise search over the whole block (ties, large k or many
    // candidates): the largest T with #{key >= T} >= k.
    int buf = 0;
    uint32_t P = 0;
    for (int bit = 30; bit >= 0; --bit) {
      const uint32_t c = P | (1u << bit);
      uint32_t mk[2];
#pragma unroll
      for (int v = 0; v < 2; ++v) {
        uint32_t x = 0;
#pragma unroll
        for (int e = 0; e < 8; ++e) x |= (uint32_t)(key_of(a[v][e]) >= c) << e;
        mk[v] = x;
      }
      const uint32_t n = wg_count<NT>(mk, l.misc + (buf ? M_RED1 : M_RED0));
      buf ^= 1;
      if ((int)n >= kq) P = c;
    }
    T = P;
    uint32_t gtm[2], eqm[2];
#pragma unroll
    for (int v = 0; v < 2; ++v) {
      uint32_t g = 0, e2 = 0;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        g |= (uint32_t)(key_of(a[v][e]) > T) << e;
        e2 |= (uint32_t)(key_of(a[v][e]) == T) << e;
      }
      gtm[v] = g;
      eqm[v] = e2;
    }
    const uint32_t ngt = wg_count<NT>(gtm, l.misc + (buf ? M_RED1 : M_RED0));
    buf ^= 1;
    const uint32_t need = (uint32_t)kq - ngt;
    uint32_t ecnt[2], ebase[2];
#pragma unroll
    for (int v = 0; v < 2; ++v) ecnt[v] = __popc(eqm[v]);
    wg_scan<NT>(ecnt, ebase, l.misc + (buf ? M_RED1 : M_RED0));
#pragma unroll
    for (int v = 0; v < 2; ++v) {
      uint32_t r = ebase[v];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        if ((eqm[v] >> e) & 1u) {
          if (r == need - 1) l.misc[M_ILAST] = eb + v * 8 + e;
          ++r;
        }
      }
    }
    lds_sync();
    i_last = sgpr(l.misc[M_ILAST]);
    notie = false;
    uint32_t scnt[2], sbase[2];
#pragma unroll
    for (int v = 0; v < 2; ++v) {
      uint32_t c = 0;
#pragma unroll
      for (int e = 0; e < 8; ++e)
        c += ((gtm[v] >> e) & 1u) || (((eqm[v] >> e) & 1u) && eb + v * 8 + e <= i_last);
      scnt[v] = c;
    }
    wg_scan<NT>(scnt, sbase, l.misc + M_RED2);
    const uint32_t row0 = (uint32_t)p.new_slot * kq;
#pragma unroll
    for (int v = 0; v < 2; ++v) {
      uint32_t pos = sbase[v];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const uint32_t i = eb + v * 8 + e;
        const bool sel = ((gtm[v] >> e) & 1u) || (((eqm[v] >> e) & 1u) && i <= i_last);
        if (sel) {
          E::store(rw, row0 + pos, E::make(i, a[v][e]));
          ++pos;
        }
      }
    }
  }

  // ---------------------------------------------- 4. e = Q(a with a[I] = 0)
  const float Tf = __uint_as_float(T);
  float x[2][8], mn[2], mx[2];
  // kept elements: |a| > T, and |a| == T up to index i_last; without ties
  // at the threshold that is |a| >= T (a workgroup-uniform case)
  if (notie) {
#pragma unroll
    for (int v = 0; v < 2; ++v)
#pragma unroll
      for (int e = 0; e < 8; ++e) x[v][e] = (__builtin_fabsf(a[v][e]) >= Tf) ? 0.0f : a[v][e];
  } else {
    // this thread's elements up to index i_last: [0, last_here]
    const int last_here = (int)i_last - (int)eb;
#pragma unroll
    for (int v = 0; v < 2; ++v)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float ab = __builtin_fabsf(a[v][e]);
        const bool kept = (ab > Tf) | ((ab == Tf) & (v * 8 + e <= last_here));
        x[v][e] = kept ? 0.0f : a[v][e];
      }
  }
#pragma unroll
  for (int v = 0; v < 2; ++v) {
    if (full) {
      mn[v] = __builtin_fminf(__builtin_fminf(__builtin_fminf(x[v][0], x[v][1]), x[v][2]),
                              __builtin_fminf(__builtin_fminf(x[v][3], x[v][4]), x[v][5]));
      mn[v] = __builtin_fminf(mn[v], __builtin_fminf(x[v][6], x[v][7]));
      mx[v] = __builtin_fmaxf(__builtin_fmaxf(__builtin_fmaxf(x[v][0], x[v][1]), x[v][2]),
                              __builtin_fmaxf(__builtin_fmaxf(x[v][3], x[v][4]), x[v][5]));
      mx[v] = __builtin_fmaxf(mx[v], __builtin_fmaxf(x[v][6], x[v][7]));
    } else {
      mn[v] = __builtin_inff();
      mx[v] = -__builtin_inff();
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (v * 8 + e < rem) { mn[v] = __builtin_fminf(mn[v], x[v][e]); mx[v] = __builtin_fmaxf(mx[v], x[v][e]); }
    }
  }
  if (!pair_buckets) {
    float lo = __builtin_fminf(mn[0], mn[1]), hi = __builtin_fmaxf(mx[0], mx[1]);
    group_minmax(lo, hi, bl - 4);
    mn[0] = mn[1] = lo;
    mx[0] = mx[1] = hi;
  }
  uint32_t w[2];
  float u[2];
#pragma unroll
  for (int v = 0; v < 2; ++v) {
    mn[v] = mn[v] + 0.0f;  // a bucket bound of -0 is stored as +0
    mx[v] = mx[v] + 0.0f;
    u[v] = div15(mx[v] - mn[v]);
  }
#pragma unroll
  for (int v = 0; v < 2; ++v) {
    // Codes from two products that bracket the quotient: v_rcp is within
    // 1 ulp for these u, so r_lo < 1/u < r_hi and
    // rint((x-min)*r_lo) <= rint((x-min)/u) <= rint((x-min)*r_hi).  Where
    // the two agree (all but a few elements in a million) the code is
    // exact; elsewhere it is recomputed with an IEEE division.
    const float uv = u[v], mnv = mn[v];
    const float rcp = __builtin_amdgcn_rcpf(uv);
    const float r_lo = __uint_as_float(__float_as_uint(rcp) - 2u);
    const float r_hi = __uint_as_float(__float_as_uint(rcp) + 2u);
    uint32_t d1e = 0, d1o = 0, d2e = 0, d2o = 0;
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      const float ye = x[v][2 * h] - mnv, yo = x[v][2 * h + 1] - mnv;
      const float p1e = ye * r_lo, p1o = yo * r_lo;
      const float p2e = ye * r_hi, p2o = yo * r_hi;
      d1e = __builtin_amdgcn_cvt_pk_u8_f32(p1e, h, d1e);  // round half to even, clamp to [0, 255]
      d1o = __builtin_amdgcn_cvt_pk_u8_f32(p1o, h, d1o);
      d2e = __builtin_amdgcn_cvt_pk_u8_f32(p2e, h, d2e);
      d2o = __builtin_amdgcn_cvt_pk_u8_f32(p2o, h, d2o);
    }
    uint32_t wv = d1e | (d1o << 4);
    const bool exact_u = uv >= 0x1p-125f && uv <= 0x1p+125f;
    if (!exact_u | (d1e != d2e) | (d1o != d2o)) {
      wv = 0;
      if (uv != 0.0f) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float y = x[v][e] - mnv;
          float rr = __builtin_rintf(y / uv);
          rr = __builtin_fminf(__builtin_fmaxf(rr, 0.0f), 15.0f);
          wv |= (uint32_t)rr << (4 * e);
        }
      }
    }
    if (!full) {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (v * 8 + e >= rem) wv &= ~(0xFu << (4 * e));
    }
    w[v] = wv;
  }
  if ((int)eb < s) {
    __builtin_amdgcn_raw_buffer_store_b64(u32x2{w[0], w[1]}, re, eb >> 1, 0, 0);
    if (pair_buckets) {
      __builtin_amdgcn_raw_buffer_store_b64(u32x2{__float_as_uint(mn[0]), __float_as_uint(mx[0])}, rs,
                                            eb, 0, 0);
      if ((int)eb + 8 < s)
        __builtin_amdgcn_raw_buffer_store_b64(u32x2{__float_as_uint(mn[1]), __float_as_uint(mx[1])}, rs,
                                              eb + 8, 0, 0);
    } else if ((eb & ((1u << bl) - 1)) == 0) {
      __builtin_amdgcn_raw_buffer_store_b64(u32x2{__float_as_uint(mn[0]), __float_as_uint(mx[0])}, rs,
                                            (eb >> bl) * 8, 0, 0);
    }
  }
}

// ============================================================ update
// z1 / z2 hold, per element of the block, sum beta1^r V and sum beta2^r V^2
// (then z1 the parameter decrement).  Element i lives at word
// ((i >> 2) & 3) * 4*NT + (i >> 4) * 4 + (i & 3), so that the 16 elements of a
// thread are four 16-byte words at a stride of 4*NT words and a wave's
// 16-byte accesses fall on consecutive addresses.  Word CAP of each array is
// a sink for lanes without an entry, which keeps the sparse updates free of
// branches.
template <int NT>
__device__ __forceinline__ uint32_t zpos(uint32_t i) {
  return ((i >> 2) & 3u) * (4u * NT) + (i >> 4) * 4u + (i & 3u);
}

// What the update kernel holds for one block before processing it: its
// geometry, its parameters and two entries per thread of its window record
// (the live rows are the record's first n_live*k_q entries).
template <bool PBF16, bool VF32>
struct UpdateBlock {
  Span g;
  Raw8<PBF16> th[2];
  typename Entry<VF32>::T w[2];
};

template <int NT, bool VF>
constexpr size_t update_lds_bytes() {
  return (size_t)2 * (NT * kLaneElems + 16) * 4 + (size_t)(2 * NT + 1) * (VF ? 8 : 4);
}

// One wave (rotating with the block) rebuilds the moments of the block's
// window entries, oldest row first, and turns them into parameter
// decrements; then every thread updates its own elements.  RUN = true: the
// blocks are full and workgroups are persistent, workgroup w taking the run
// of blocks first_block + [w*per, (w+1)*per) and loading the next block's
// parameters and window entries before it processes the current one.
// RUN = false: workgroup w takes block first_block + w alone.  EXPORT = true
// writes dense m-hat and v-hat instead of updating theta.
// LDS (about 35 KB per workgroup) allows 4 workgroups per compute unit, one
// wave of each per SIMD; telling the compiler so lets it keep independent LDS
// reads in flight together instead of minimising registers.
template <int NT, bool PBF16, bool VF32, bool EXPORT, bool RUN, int KC>
__global__ void __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(4))) update_kernel(StepParams p, int64_t first_block, int64_t num_blocks,
                                                    int64_t per, float* mhat, float* vhat) {
  constexpr int NW = NT / kWave;
  constexpr int CAP = NT * kLaneElems;
  constexpr int kChunks = KC;              // 64-entry window chunks the leader holds
  using E = Entry<VF32>;
  using ET = typename E::T;
  using UB = UpdateBlock<PBF16, VF32>;
  extern __shared__ __align__(16) uint32_t smem[];
  float* const z1 = (float*)smem;
  float* const z2 = z1 + CAP + 16;
  // [2*NT] live window entries, then one entry that is always empty
  ET* const stage = (ET*)(z2 + CAP + 16);

  const int tid = thread_id(), lane = tid & (kWave - 1), wave = (int)sgpr(tid / kWave);
  const uint32_t eb = (uint32_t)tid * kLaneElems;
  const int m = p.window, n_live = p.n_live;
  // oldest live row first: the row written at step s is slot (s-1) mod m
  const int slot0 = (p.new_slot + 1 + m - n_live) % m;
  const float w1s = lane < kMaxWindow ? constant_ptr(p.wpow)[lane] : 0.0f;
  const float w2s = lane < kMaxWindow ? constant_ptr(p.wpow)[kMaxWindow + lane] : 0.0f;

  // this thread's 16 words of each accumulator
  auto zero_own = [&](float* a1, float* a2) {
    const float4 zero = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      *(float4*)(a1 + q * 4 * NT + tid * 4) = zero;
      *(float4*)(a2 + q * 4 * NT + tid * 4) = zero;
    }
  };
  if (tid == 0) stage[2 * NT] = E::none();
  if (RUN) zero_own(z1, z2);
  Cursor cursor = {0, 0, 0};
  auto fetch = [&](int32_t gb, UB& u) {
    u.g = RUN ? seek_full(p, cursor, gb, PBF16 ? 2 : 4) : span_of(p, gb, PBF16 ? 2 : 4);
    // unconditional loads keep the count of loads in flight fixed; entries
    // past the record read 0 and entries past the live rows are not used
    const Rsrc rw = window_rsrc<VF32 ? 2 : 1>(p, gb, u.g.kq);
    u.w[0] = E::load(rw, tid);
    u.w[1] = E::load(rw, tid + NT);
    if (!EXPORT) {
      const Rsrc rp = make_rsrc((const void*)u.g.base, vec_bytes<PBF16>(u.g.s));
#pragma unroll
      for (int v = 0; v < 2; ++v) u.th[v] = load8<PBF16>(rp, eb + v * 8);
    }
  };

  auto process = [&](const UB& u) {
    const int s = u.g.s, kq = u.g.kq;
    const int leader = u.g.gb & (NW - 1);
    const int R = (kq + kWave - 1) / kWave;
    const bool staged = n_live * kq <= 2 * NT && n_live * R <= kChunks;
    // In a run the accumulators are clean when a block starts: the θ pass
    // clears z1 behind it and the leader clears the z2 words it used.  A
    // workgroup that takes one block starts from uninitialised LDS.
    if (!RUN) zero_own(z1, z2);
    stage[tid] = u.w[0];
    stage[tid + NT] = u.w[1];
    lds_sync();

    if (wave == leader) {
      auto step_of = [&](float s1, float s2) {
        const float mh = p.c1 * s1;
        const float vh = p.c2 * s2;
        const float den = p.eps + __builtin_amdgcn_sqrtf(vh);
        return p.lr * (mh * __builtin_amdgcn_rcpf(den));
      };
      if (staged) {
        // Chunk c: row c / R in age order (slot (slot0 + row) mod m), entries
        // (c mod R)*64 + lane.  All kChunks chunks are processed without
        // branches: chunks past the live rows read the empty entry, and
        // lanes without an entry work on the sink word.
        const int nch = opaque(n_live * R);
        uint32_t zp[kChunks];
        float val[kChunks];
        int rr[kChunks];
        {
          int row = 0, col = 0, slot = slot0;
#pragma unroll
          for (int c = 0; c < kChunks; ++c) {
            const int jj = col * kWave + lane;
            const ET x = stage[(c < nch && jj < kq) ? slot * kq + jj : 2 * NT];
            const uint32_t i = E::idx(x);
            zp[c] = i < (uint32_t)s ? zpos<NT>(i) : (uint32_t)CAP;
            val[c] = E::val(x);
            rr[c] = (n_live - 1 - row) & (kMaxWindow - 1);
            if (++col == R) {
              col = 0;
              ++row;
              if (++slot == m) slot = 0;
            }
          }
        }
        // the entries of one row (or of one 64-entry part of it) have
        // distinct indices, so each chunk reads, adds and writes back its
        // words (the sink word's lanes race harmlessly); chunks follow each
        // other oldest row first
#pragma unroll
        for (int c = 0; c < kChunks; ++c) {
          const float w1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(w1s), rr[c]));
          const float w2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(w2s), rr[c]));
          const float v = val[c];
          const float x1 = w1 * v;
          const float vv = v * v;
          const float x2 = w2 * vv;
          const float a1 = z1[zp[c]], a2 = z2[zp[c]];
          z1[zp[c]] = a1 + x1;
          z2[zp[c]] = a2 + x2;
        }
        if (!EXPORT) {
          // every entry's sums are read before any word is overwritten, so an
          // index that occurs in several rows gets the same decrement from
          // each occurrence
          float d[kChunks];
#pragma unroll
          for (int c = 0; c < kChunks; ++c) d[c] = step_of(z1[zp[c]], z2[zp[c]]);
#pragma unroll
          for (int c = 0; c < kChunks; ++c) {
            z1[zp[c]] = d[c];
            z2[zp[c]] = 0.0f;
          }
        }
      } else {
        const Rsrc rw = window_rsrc<VF32 ? 2 : 1>(p, u.g.gb, kq);
        for (int row = 0, slot = slot0; row < n_live; ++row, slot = (slot + 1 == m) ? 0 : slot + 1) {
          const int r = n_live - 1 - row;
          const float w1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(w1s), r));
          const float w2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(w2s), r));
          for (int jj = lane; jj < kq; jj += kWave) {
            const ET x = E::load(rw, slot * kq + jj);
            const uint32_t i = E::idx(x);
            const uint32_t zp = i < (uint32_t)s ? zpos<NT>(i) : (uint32_t)CAP;
            const float v = E::val(x);
            const float vv = v * v;
            const float x1 = w1 * v, x2 = w2 * vv;
            const float a1 = z1[zp], a2 = z2[zp];
            z1[zp] = a1 + x1;
            z2[zp] = a2 + x2;
          }
        }
        if (!EXPORT) {
          // one 64-entry chunk at a time; z2 = -1 marks a converted word
          for (int row = 0, slot = slot0; row < n_live; ++row, slot = (slot + 1 == m) ? 0 : slot + 1)
            for (int jj = lane; jj < kq; jj += kWave) {
              const uint32_t i = E::idx(E::load(rw, slot * kq + jj));
              if (i < (uint32_t)s) {
                const uint32_t zp = zpos<NT>(i);
                const float s2 = z2[zp];
                if (s2 >= 0.0f) {
                  z1[zp] = step_of(z1[zp], s2);
                  z2[zp] = -1.0f;
                }
              }
            }
        }
      }
    }
    lds_sync();

    if (EXPORT) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const float4 s1 = *(const float4*)(z1 + q * 4 * NT + tid * 4);
        const float4 s2 = *(const float4*)(z2 + q * 4 * NT + tid * 4);
        const float a1[4] = {s1.x, s1.y, s1.z, s1.w}, a2[4] = {s2.x, s2.y, s2.z, s2.w};
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const uint32_t i = eb + q * 4 + r;
          if ((int)i < s) {
            mhat[u.g.e0 + i] = p.c1 * a1[r];
            vhat[u.g.e0 + i] = p.c2 * a2[r];
          }
        }
      }
      return;
    }

    // ---------------------------------------------- 6. parameter update
    const bool full = s == NT * kLaneElems;
    const Rsrc rp = make_rsrc((const void*)u.g.base, vec_bytes<PBF16>(s));
#pragma unroll
    for (int v = 0; v < 2; ++v) {
      const uint32_t e0 = eb + v * 8;   // vectors past s store nothing
      const float4 u0 = *(const float4*)(z1 + (2 * v) * 4 * NT + tid * 4);
      const float4 u1 = *(const float4*)(z1 + (2 * v + 1) * 4 * NT + tid * 4);
      if (RUN) {
        // clear behind the read; the unstaged path leaves marks in z2 too
        const float4 zero = make_float4(0.f, 0.f, 0.f, 0.f);
        *(float4*)(z1 + (2 * v) * 4 * NT + tid * 4) = zero;
        *(float4*)(z1 + (2 * v + 1) * 4 * NT + tid * 4) = zero;
        if (!staged) {
          *(float4*)(z2 + (2 * v) * 4 * NT + tid * 4) = zero;
          *(float4*)(z2 + (2 * v + 1) * 4 * NT + tid * 4) = zero;
        }
      }
      const float upd[8] = {u0.x, u0.y, u0.z, u0.w, u1.x, u1.y, u1.z, u1.w};
      float thf[8], out[8];
      unpack8<PBF16>(u.th[v], thf);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float base = p.decay_is_one ? thf[e] : thf[e] * p.decay;
        out[e] = base - upd[e];
      }
      // a full block holds whole threads (B_d is a multiple of 16)
      if (RUN) {
        if ((int)eb < s) store8<PBF16>(rp, e0, s, true, out);
      } else {
        store8<PBF16>(rp, e0, s, full, out);
      }
    }
  };

  // Two register sets take turns, and the next block is always fetched (the
  // last block of a run fetches itself again), so that the count of loads
  // issued after any block's data is fixed and the waits for that data let
  // the next block's loads stay in flight.
  if (!RUN) {
    UB A;
    fetch((int32_t)(first_block + block_id()), A);
    process(A);
    return;
  }
  const int32_t nb = (int32_t)num_blocks, run = (int32_t)per;
  const int32_t lo = (int32_t)block_id() * run;
  if (lo >= nb) return;
  const int32_t g0 = (int32_t)first_block;
  const int32_t hi = g0 + (lo + run < nb ? lo + run : nb);
  int32_t g = g0 + lo;
  UB A, B;
  fetch(g, A);
  for (;;) {
    const int32_t g1 = g + 1;
    const bool m1 = g1 < hi;
    fetch(m1 ? g1 : g, B);
    process(A);
    if (!m1) break;
    const int32_t g2 = g1 + 1;
    const bool m2 = g2 < hi;
    fetch(m2 ? g2 : g1, A);
    process(B);
    if (!m2) break;
    g = g2;
  }
}


// Resident workgroups of one update launch: enough to fill every compute
// unit, computed once per device.
template <int NT, bool PB, bool VF>
int64_t update_grid(size_t lds) {
  static int64_t cache[64] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 1024;
  if (!cache[dev]) {
    int per_cu = 0, cus = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, update_kernel<NT, PB, VF, false, true, 16>, NT, lds) !=
            hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        per_cu < 1 || cus < 1)
      return 1024;
    cache[dev] = (int64_t)per_cu * cus;
  }
  return cache[dev];
}

template <int NT, bool GB, bool VF>
hipError_t launch_select_t(const StepParams& p, hipStream_t stream) {
  const size_t lds = SelectLds<NT>::words() * 4;
  hipLaunchKernelGGL((select_kernel<NT, GB, VF>), dim3((uint32_t)p.total_blocks), dim3(NT), lds, stream, p);
  return hipGetLastError();
}

// Chunks of 64 window entries the update's leader wave processes per block:
// the live rows of a full block rounded up to 4, 8, 10, 12 or 16.
inline int chunk_class(const StepParams& p) {
  const int R = (p.k_full + kWave - 1) / kWave;
  const int nch = p.n_live * R;
  return nch <= 4 ? 4 : nch <= 8 ? 8 : nch <= 10 ? 10 : nch <= 12 ? 12 : 16;
}

template <int NT, bool PB, bool VF, int KC>
void launch_update_run(const StepParams& p, int64_t grid, int64_t per, size_t lds, hipStream_t stream) {
  hipLaunchKernelGGL((update_kernel<NT, PB, VF, false, true, KC>), dim3((uint32_t)grid), dim3(NT), lds, stream, p,
                     (int64_t)0, p.n_full, per, (float*)nullptr, (float*)nullptr);
}

// The full blocks [0, n_full) in persistent runs, then the ragged blocks one
// workgroup each.
template <int NT, bool PB, bool VF>
hipError_t launch_update_t(const StepParams& p, hipStream_t stream) {
  const size_t lds = update_lds_bytes<NT, VF>();
  if (p.n_full > 0) {
    int64_t grid = update_grid<NT, PB, VF>(lds);
    if (grid > p.n_full) grid = p.n_full;
    const int64_t per = (p.n_full + grid - 1) / grid;
    grid = (p.n_full + per - 1) / per;
    switch (chunk_class(p)) {
      case 4: launch_update_run<NT, PB, VF, 4>(p, grid, per, lds, stream); break;
      case 8: launch_update_run<NT, PB, VF, 8>(p, grid, per, lds, stream); break;
      case 10: launch_update_run<NT, PB, VF, 10>(p, grid, per, lds, stream); break;
      case 12: launch_update_run<NT, PB, VF, 12>(p, grid, per, lds, stream); break;
      default: launch_update_run<NT, PB, VF, 16>(p, grid, per, lds, stream); break;
    }
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const int64_t tails = p.total_blocks - p.n_full;
  if (tails > 0) {
    hipLaunchKernelGGL((update_kernel<NT, PB, VF, false, false, 16>), dim3((uint32_t)tails), dim3(NT), lds, stream,
                       p, p.n_full, tails, (int64_t)1, (float*)nullptr, (float*)nullptr);
    return hipGetLastError();
  }
  return hipSuccess;
}

template <int NT, bool VF>
hipError_t launch_export(const StepParams& p, int64_t first_block, int64_t blocks, float* mh, float* vh,
                         hipStream_t stream) {
  const size_t lds = update_lds_bytes<NT, VF>();
  hipLaunchKernelGGL((update_kernel<NT, false, VF, true, false, 16>), dim3((uint32_t)blocks), dim3(NT), lds, stream,
                     p, first_block, blocks, (int64_t)1, mh, vh);
  return hipGetLastError();
}

}  // namespace

size_t step_lds_bytes(int block, int k_full, int value_f32) {
  (void)k_full;
  (void)value_f32;
  const int nt = threads_for_block(block);
  const size_t sel = (nt == 64 ? SelectLds<64>::words() : SelectLds<256>::words()) * 4;
  const size_t upd = nt == 64 ? update_lds_bytes<64, true>() : update_lds_bytes<256, true>();
  return sel > upd ? sel : upd;
}

hipError_t launch_select(const StepParams& p, int grad_bf16, int value_f32, hipStream_t stream) {
  if (threads_for_block(p.block) == 64) {
    if (grad_bf16) return value_f32 ? launch_select_t<64, true, true>(p, stream) : launch_select_t<64, true, false>(p, stream);
    return value_f32 ? launch_select_t<64, false, true>(p, stream) : launch_select_t<64, false, false>(p, stream);
  }
  if (grad_bf16) return value_f32 ? launch_select_t<256, true, true>(p, stream) : launch_select_t<256, true, false>(p, stream);
  return value_f32 ? launch_select_t<256, false, true>(p, stream) : launch_select_t<256, false, false>(p, stream);
}

hipError_t launch_update(const StepParams& p, int param_bf16, int value_f32, hipStream_t stream) {
  if (threads_for_block(p.block) == 64) {
    if (param_bf16) return value_f32 ? launch_update_t<64, true, true>(p, stream) : launch_update_t<64, true, false>(p, stream);
    return value_f32 ? launch_update_t<64, false, true>(p, stream) : launch_update_t<64, false, false>(p, stream);
  }
  if (param_bf16) return value_f32 ? launch_update_t<256, true, true>(p, stream) : launch_update_t<256, true, false>(p, stream);
  return value_f32 ? launch_update_t<256, false, true>(p, stream) : launch_update_t<256, false, false>(p, stream);
}

hipError_t launch_moments(const StepParams& p, int64_t first_block, int64_t num_blocks, float* mhat,
                          float* vhat, int value_f32, hipStream_t stream) {
  if (threads_for_block(p.block) == 64)
    return value_f32 ? launch_export<64, true>(p, first_block, num_blocks, mhat, vhat, stream)
                     : launch_export<64, false>(p, first_block, num_blocks, mhat, vhat, stream);
  return value_f32 ? launch_export<256, true>(p, first_block, num_blocks, mhat, vhat, stream)
                   : launch_export<256, false>(p, first_block, num_blocks, mhat, vhat, stream);
}

}  // namespace microadam
