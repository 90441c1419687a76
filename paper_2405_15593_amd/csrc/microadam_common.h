// Device-side building blocks shared by the MicroAdam step kernels for CDNA4
// (gfx950): wave operations, buffer resources, element vectors, window
// entries, block geometry, and the per-lane parts of the select (decode,
// quantization, codes).  Internal to the library.
//
// Arithmetic that decides an integer (EF decode, accumulator, Top-K order,
// bucket min/max, codes) is binary32 with one rounding per written operation
// (the sources are compiled with -ffp-contract=off); the only fused operations
// in that part are in div15, which is exact, and the code brackets of
// vector_codes, which are checked against the exact quotient's rounding.  The
// device code is compiled without IEEE NaN handling (min/max do not quiet
// NaNs): gradients are taken to be finite.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "microadam_device.h"

namespace microadam {
namespace {

constexpr int kWave = 64;

// A compile-time flag passed to generic lambdas (branches chosen once, not
// per element).
template <bool B>
struct BoolTag {
  static constexpr bool value = B;
};
constexpr int kLaneElems = 16;       // consecutive elements per thread
constexpr uint32_t kNoEntry = 0xFFFFFFFFu;

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef __amdgpu_buffer_rsrc_t Rsrc;

// ---------------------------------------------------------------- wave ops
__device__ __forceinline__ uint64_t ballot(bool p) { return __ballot(p); }
__device__ __forceinline__ uint32_t lanes_below(uint64_t m) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}
// base + the number of lanes below this one in m
__device__ __forceinline__ uint32_t lanes_below_from(uint64_t m, uint32_t base) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)m, base));
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
// The same for a per-lane value: comparisons against it are made where
// written (in the branch that needs them), not once for every branch.
__device__ __forceinline__ int opaque_v(int x) {
  asm volatile("" : "+v"(x));
  return x;
}
// A uniform float the compiler must treat as new: comparisons against it in
// different loops are not merged and kept alive between them.
__device__ __forceinline__ float opaque_f(float x) {
  int b = __builtin_amdgcn_readfirstlane(__float_as_int(x));
  asm volatile("" : "+s"(b));
  return __int_as_float(b);
}
// Work-item and workgroup ids straight from the hardware registers (the
// library wrappers behind threadIdx / blockIdx are not inlined into code
// built without IEEE mode).
__device__ __forceinline__ int thread_id() { return (int)__builtin_amdgcn_workitem_id_x(); }
__device__ __forceinline__ int64_t block_id() { return (int64_t)__builtin_amdgcn_workgroup_id_x(); }

// Block handled by workgroup w of a launch over n blocks.  Workgroups are
// dispatched to the eight XCDs (each with its own L2) in turn, so XCD x runs
// w = x, x + 8, x + 16, ...; this gives each XCD one contiguous range of
// blocks instead (a bijection of [0, n)): neighbouring blocks, whose state
// records may share cache lines, then meet in the same L2.
#ifndef MICROADAM_XCD_MAP
#define MICROADAM_XCD_MAP 1
#endif
__device__ __forceinline__ int64_t xcd_block(int64_t w, int64_t n) {
  if (!MICROADAM_XCD_MAP) return w;
  const int64_t x = w & 7, j = w >> 3, q = n >> 3, r = n & 7;
  return x * q + (x < r ? x : r) + j;
}

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

// Error-feedback code formats (a template parameter of the select kernel):
// bit 0: 8-bit codes, one byte per element (else 4-bit, two per byte);
// bit 1: randomized rounding (Lemma 1) instead of round-to-nearest.
constexpr int kEf8 = 1, kEfRandom = 2;

// Philox4x32-10 (Salmon, Moraes, Dror and Shaw, "Parallel Random Numbers: As
// Easy as 1, 2, 3", SC 2011): ten rounds of two 32x32 -> 64-bit products
// with the round keys; the key advances by the Weyl constants between rounds
// (the key words are wave-uniform and stay in scalar registers).
__device__ __forceinline__ u32x4 philox4x32_10(u32x4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r > 0) {
      k0 += 0x9E3779B9u;
      k1 += 0xBB67AE85u;
    }
    // one 32x32 -> 64-bit multiply each (v_mad_u64_u32)
    const uint64_t p0 = (uint64_t)0xD2511F53u * c[0];
    const uint64_t p1 = (uint64_t)0xCD9E8D57u * c[2];
    c = u32x4{(uint32_t)(p1 >> 32) ^ c[1] ^ k0, (uint32_t)p1, (uint32_t)(p0 >> 32) ^ c[3] ^ k1, (uint32_t)p0};
  }
  return c;
}

// Randomized code (Lemma 1): floor(y + xi) for y = (x - lo)/u (IEEE
// division) and xi = w24 * 2^-24, taken exactly: floor(y) + 1 when w24 +
// floor(2^24 * frac(y)) >= 2^24 (the fraction and its scaling are exact);
// clamped to [0, L].  u != 0.
__device__ __forceinline__ uint32_t code_randomized(float x, float lo, float u, float levels, uint32_t w24) {
  const float y = (x - lo) / u;
  const float fy = __builtin_floorf(y);
  const float f = y - fy;
  const uint32_t fr = (uint32_t)__builtin_floorf(f * 16777216.0f);
  float r = fy + ((w24 + fr >= (1u << 24)) ? 1.0f : 0.0f);
  r = __builtin_fminf(__builtin_fmaxf(r, 0.0f), levels);
  return (uint32_t)r;
}

// Round-to-nearest code (Algorithm 2, Q): rint((x - lo)/u) with an IEEE
// division, clamped to [0, L].  u != 0.
__device__ __forceinline__ uint32_t code_nearest(float x, float lo, float u, float levels) {
  const float r = __builtin_rintf((x - lo) / u);
  return (uint32_t)__builtin_fminf(__builtin_fmaxf(r, 0.0f), levels);
}

// Quantization step of a bucket: (max - min) / L, correctly rounded.
template <int EFM>
__device__ __forceinline__ float ef_step(float d) {
  if constexpr (EFM & kEf8) return d / 255.0f;
  else return div15(d);
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

// Two floats rounded to bf16 (half to even), lo in the low half: one
// v_cvt_pk_bf16_f32 for the pair.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  typedef float f32x2_t __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){lo, hi}, bf16x2_t));
}

// 2w + c: the lane's flag c shifted into the low bit of w, by one add with
// carry that takes c from the wave's lane mask m (a per-lane bit set in one
// instruction per element).  The two wait states ahead of the add cover a
// mask written by the instruction just before it.  A flag that is a logical
// combination of compares is best passed as the same combination of their
// masks (shift_in_mask): a ballot of the combined flag costs two more
// instructions per element.
__device__ __forceinline__ uint32_t shift_in_mask(uint32_t w, uint64_t m) {
  uint32_t r;
  uint64_t carry_out;
  asm("s_nop 1\n\tv_addc_co_u32_e64 %0, %1, %2, %2, %3" : "=v"(r), "=s"(carry_out) : "v"(w), "s"(m));
  return r;
}
__device__ __forceinline__ uint32_t shift_in_flag(uint32_t w, bool c) {
  return shift_in_mask(w, __builtin_amdgcn_ballot_w64(c));
}
// shift_in_mask, and x replaced by 0 in the lanes of m, from the one mask.
__device__ __forceinline__ uint32_t shift_in_mask_zero(uint32_t w, uint64_t m, float& x) {
  uint32_t r;
  uint64_t carry_out;
  asm("s_nop 1\n\tv_addc_co_u32_e64 %0, %1, %3, %3, %4\n\tv_cndmask_b32_e64 %2, %2, 0, %4"
      : "=&v"(r), "=&s"(carry_out), "+v"(x)
      : "v"(w), "s"(m));
  return r;
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
  r.first_bucket = d->first_bucket;
  r.num_buckets = d->num_buckets;
  r.ragged_before = d->ragged_before;
  r.reserved = 0;
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
      for (int h = 0; h < 4; ++h) w[h] = pack_bf16x2(in[2 * h], in[2 * h + 1]);
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

// ------------------------------------------------ streamed 16-byte vectors
// Cache policy of the accesses that stream through a step once (parameters,
// gradients, codes, bucket pairs, window records): nt, bit 1 of the buffer
// instructions' cache-policy operand.  Measured on MI355X with coalesced
// accesses (every 16-byte access of a wave in one contiguous 1 KB run), nt on
// both the loads and the stores of a pattern moves it 10-11% faster (a
// parameter read-modify-write with window reads: 5.17 -> 4.71 ms per 29.65 GB;
// the select's reads and writes: 4.16 -> 3.83 ms per 22.17 GB); with each
// lane's accesses 128 bytes apart it is slower instead (4.25 -> 7.6 ms), so
// it goes only on coalesced accesses, and not on lines that another wave
// reads soon after (the large-block update's row segments).
constexpr int kStream = 2;

// A thread's 16 elements of a block as 16-byte vectors that consecutive
// threads take in turn: vector v of thread t holds the EV elements from
// v*EV*NT + t*EV (EV = 8 for bf16, 4 for binary32), so each vector access of
// a wave covers one contiguous kilobyte.
template <bool BF16> struct Vec16 {
  static constexpr int EV = BF16 ? 8 : 4;  // elements per vector
  static constexpr int NV = kLaneElems / EV;  // vectors per thread
  template <int NT>
  __device__ static uint32_t first(int v, int t) { return (uint32_t)(v * EV * NT + t * EV); }
  __device__ static u32x4 load(Rsrc r, uint32_t elem) {
    return __builtin_amdgcn_raw_buffer_load_b128(r, elem * (BF16 ? 2u : 4u), 0, kStream);
  }
  __device__ static void unpack(u32x4 x, float (&out)[EV]) {
    if constexpr (BF16) {
#pragma unroll
      for (int h = 0; h < 4; ++h) { out[2 * h] = bf16_lo(x[h]); out[2 * h + 1] = bf16_hi(x[h]); }
    } else {
#pragma unroll
      for (int h = 0; h < 4; ++h) out[h] = __uint_as_float(x[h]);
    }
  }
  // Stores the vector at elem: whole when `full` (workgroup-uniform), else
  // only its elements below s.
  __device__ static void store(Rsrc r, uint32_t elem, int s, bool full, const float (&in)[EV]) {
    if (full) {
      u32x4 w;
#pragma unroll
      for (int h = 0; h < 4; ++h)
        w[h] = BF16 ? pack_bf16x2(in[2 * h], in[2 * h + 1]) : __float_as_uint(in[h]);
      __builtin_amdgcn_raw_buffer_store_b128(w, r, elem * (BF16 ? 2u : 4u), 0, kStream);
    } else {
#pragma unroll
      for (int e = 0; e < EV; ++e) {
        if ((int)elem + e < s) {
          if constexpr (BF16) __builtin_amdgcn_raw_buffer_store_b16((uint16_t)to_bf16_bits(in[e]), r, (elem + e) * 2, 0, 0);
          else __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(in[e]), r, (elem + e) * 4, 0, 0);
        }
      }
    }
  }
};

// ------------------------------------------------------- window entries
// bf16 values: one word (index | bf16 << 16); f32 values: (index, value).
template <bool VF32> struct Entry {
  typedef typename std::conditional<VF32, u32x2, uint32_t>::type T;
  // an entry number whose byte offset lies past every record (a buffer
  // load there reads 0)
  static constexpr uint32_t kFar = VF32 ? 0x1FFFFFFEu : 0x3FFFFFFEu;
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
  // the entry with its index replaced by w (an accumulator word, < 2^16)
  __device__ static T with_word(T e, uint32_t w) {
    if constexpr (VF32) return u32x2{w, e[1]};
    else return (e & 0xFFFF0000u) | w;
  }
  __device__ static uint32_t word(T e) {
    if constexpr (VF32) return e[0];
    else return e & 0xFFFFu;
  }
  template <int AUX = 0>
  __device__ static T load(Rsrc r, uint32_t entry) {
    if constexpr (VF32) return __builtin_amdgcn_raw_buffer_load_b64(r, entry * 8, 0, AUX);
    else return __builtin_amdgcn_raw_buffer_load_b32(r, entry * 4, 0, AUX);
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
  uint32_t j;             // tensor number
};

// The tensor of global block gb: from the block table, or, without one, by
// binary search over the tensor table (full blocks are numbered tensor by
// tensor, so gb < n_full lies in the last tensor whose full blocks start at
// or before it; ragged block gb - n_full belongs to the last tensor with at
// most that many ragged tensors before it).
__device__ __forceinline__ uint32_t tensor_of_block(const StepParams& p, int64_t gb) {
  if (p.block_tensor) return constant_ptr(p.block_tensor)[gb];
  const __attribute__((address_space(4))) TensorDesc* td = constant_ptr(p.tensors);
  int lo = 0, hi = p.n_tensors - 1;
  if (gb < p.n_full) {
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (td[mid].first_block <= gb) lo = mid;
      else hi = mid - 1;
    }
  } else {
    const int64_t r = gb - p.n_full;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if ((int64_t)td[mid].ragged_before <= r) lo = mid;
      else hi = mid - 1;
    }
  }
  return (uint32_t)lo;
}

__device__ __forceinline__ Block locate(const StepParams& p, int64_t gb) {
  Block b;
  const uint32_t j = tensor_of_block(p, gb);
  b.desc = load_desc(constant_ptr(p.tensors) + j);
  const bool last = (int32_t)gb == (int32_t)b.desc.last_block;
  const int32_t q = last ? (int32_t)b.desc.num_blocks - 1 : (int32_t)(gb - b.desc.first_block);
  b.e0 = (int64_t)q * p.block;
  b.s = last ? b.desc.s_last : p.block;
  b.kq = last ? b.desc.k_last : b.desc.k_full;
  b.j = j;
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
  return make_rsrc(p.state + p.win_plane + (uint64_t)gb * p.win_stride, (uint32_t)(p.window * kq * EW * 4));
}

// ============================================================ select
// One wave per block.  Lane l owns the EPL consecutive elements
// [l*EPL, (l+1)*EPL) of the block as NV = EPL/8 vectors of 8 (EPL = 16, 32
// or 64 for B_d up to 1024, 2048, 4096); lanes past the block hold no
// elements.  A wave needs no barrier: its LDS traffic is ordered by
// wave_sync alone.
//
// Top-K (Section 3.1) in three stages:
//   1. a lower bound L on the k-th largest |a|: the largest 13-bit prefix
//      value with at least k of the 128 half-lane maxima above it (each such
//      half lane holds an element >= L, so at least k elements are >= L);
//   2. the vectors holding some |a| >= L are gathered in LDS, and their
//      elements >= L (the candidates, in element order) compacted;
//   3. the k-th largest key among the candidates, bit by bit from the top.
// Blocks where a stage overflows its LDS (or k > 128) take an exact bitwise
// search over all elements instead.
constexpr int kMaxCandVec = 128;   // candidate vectors gathered in LDS
constexpr int kCandMax = 256;      // candidate elements resolved

constexpr int kRowBufWords = 320;  // the new row's 128-byte lines: k <= 128 entries of <= 8 bytes, + 2 lines

__host__ __device__ constexpr size_t select_lds_words() {
  return (size_t)kMaxCandVec * 9 + 2 * kCandMax + kRowBufWords;
}

// Orders the LDS accesses of one wave (each lane's writes before the other
// lanes' later reads); LDS operations of a wave execute in order, so this
// is only a compiler barrier and a wait for the wave's own LDS operations.
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront", "local");
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0)
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront", "local");
}

// Exclusive prefix over lanes (lane order) of a per-lane count below 16,
// and the wave total.
__device__ __forceinline__ uint32_t lane_prefix(uint32_t c, uint32_t& total) {
  uint32_t pre = 0, tot = 0;
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    const uint64_t m = ballot((c >> b) & 1u);
    pre += lanes_below(m) << b;
    tot += popc(m) << b;
  }
  total = tot;
  return pre;
}

// ------------------------------------------------ select: one lane's part
// A lane (thread) of a select kernel owns the EPL consecutive elements
// [eb, eb + EPL) of its block as NV = EPL/8 vectors of 8.  LB: its buckets
// are the lane or groups of lanes (B_q >= EPL); else buckets of whole
// vectors inside the lane.
template <int EPL, bool LB, bool GBF16, int EFM = 0>
struct LaneIn {
  static constexpr int NV = EPL / 8;
  static constexpr int CW = (EFM & kEf8) ? 2 : 1;  // code words per vector
  u32x2 st[LB ? 1 : NV];  // bucket (min, max) pairs: one, or one per vector
  uint32_t cw[NV * CW];   // codes of vector v: 4-bit, element e in bits [4e, 4e + 4)
                          // of word v; 8-bit, byte e & 3 of word 2v + e/4
  Raw8<GBF16> graw[NV];   // gradient
};

// Code values of vector v as floats (4-bit: nibbles, 8-bit: bytes).
template <int EFM>
__device__ __forceinline__ void unpack_codes(const uint32_t* cw, int v, float (&c)[8]) {
  if constexpr (EFM & kEf8) {
    const uint32_t w0 = cw[2 * v], w1 = cw[2 * v + 1];
    c[0] = ubyte<0>(w0); c[1] = ubyte<1>(w0); c[2] = ubyte<2>(w0); c[3] = ubyte<3>(w0);
    c[4] = ubyte<0>(w1); c[5] = ubyte<1>(w1); c[6] = ubyte<2>(w1); c[7] = ubyte<3>(w1);
  } else {
    const uint32_t ev = cw[v] & 0x0F0F0F0Fu, od = (cw[v] >> 4) & 0x0F0F0F0Fu;
    c[0] = ubyte<0>(ev); c[2] = ubyte<1>(ev); c[4] = ubyte<2>(ev); c[6] = ubyte<3>(ev);
    c[1] = ubyte<0>(od); c[3] = ubyte<1>(od); c[5] = ubyte<2>(od); c[7] = ubyte<3>(od);
  }
}

// Bucket pairs and codes of the lane.  `wide`: 16-byte code accesses (the
// block fills every lane of the kernel), else 8-byte ones (B_d is a multiple
// of 16, so no access then straddles the end of the block's codes).
template <int EPL, bool LB, bool GBF16, int EFM>
__device__ __forceinline__ void lane_load_codes(LaneIn<EPL, LB, GBF16, EFM>& in, Rsrc re, uint32_t eb, bool wide) {
  constexpr int NV = EPL / 8;
  if constexpr (EFM & kEf8) {
    // 16 codes per 16-byte access; B_d is a multiple of 16, so an access lies
    // wholly inside or wholly past the block's codes
#pragma unroll
    for (int q = 0; q < NV / 2; ++q) {
      const u32x4 t = __builtin_amdgcn_raw_buffer_load_b128(re, eb + 16 * q, 0, 0);
#pragma unroll
      for (int h = 0; h < 4; ++h) in.cw[4 * q + h] = t[h];
    }
  } else if (NV > 2 && wide) {
#pragma unroll
    for (int q = 0; q < NV / 4; ++q) {
      const u32x4 t = __builtin_amdgcn_raw_buffer_load_b128(re, (eb >> 1) + 16 * q, 0, 0);
#pragma unroll
      for (int h = 0; h < 4; ++h) in.cw[4 * q + h] = t[h];
    }
  } else {
#pragma unroll
    for (int q = 0; q < NV / 2; ++q) {
      const u32x2 t = __builtin_amdgcn_raw_buffer_load_b64(re, (eb >> 1) + 8 * q, 0, 0);
      in.cw[2 * q] = t[0];
      in.cw[2 * q + 1] = t[1];
    }
  }
}

template <int EPL, bool LB, bool GBF16, int EFM>
__device__ __forceinline__ void lane_load_state(LaneIn<EPL, LB, GBF16, EFM>& in, Rsrc re, Rsrc rs, uint32_t eb,
                                                int bl, bool wide) {
  constexpr int NV = EPL / 8;
#pragma unroll
  for (int v = 0; v < (LB ? 1 : NV); ++v)
    in.st[v] = __builtin_amdgcn_raw_buffer_load_b64(rs, ((eb + 8 * v) >> bl) * 8, 0, 0);
  lane_load_codes(in, re, eb, wide);
}

template <int EPL, bool LB, bool GBF16, int EFM>
__device__ __forceinline__ void lane_load_grad(LaneIn<EPL, LB, GBF16, EFM>& in, Rsrc rg, uint32_t eb) {
#pragma unroll
  for (int v = 0; v < EPL / 8; ++v) in.graw[v] = load8<GBF16>(rg, eb + 8 * v);
}

// a = g + Q^-1(e) (Algorithm 1; Algorithm 2, Q^-1).  rem: the lane's
// elements below the end of the block, [0, rem); the others are 0.
template <int EPL, bool LB, bool GBF16, int EFM>
__device__ __forceinline__ void lane_decode(const LaneIn<EPL, LB, GBF16, EFM>& in, float (&a)[EPL / 8][8], int rem,
                                            bool full) {
  constexpr int NV = EPL / 8;
  {
    float lo0 = 0.0f, u0 = 0.0f;
    if constexpr (LB) {
      lo0 = __uint_as_float(in.st[0][0]);
      u0 = ef_step<EFM>(__uint_as_float(in.st[0][1]) - lo0);
    }
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const float lo = LB ? lo0 : __uint_as_float(in.st[v][0]);
      const float u = LB ? u0 : ef_step<EFM>(__uint_as_float(in.st[v][1]) - lo);
      float g[8], c[8];
      unpack8<GBF16>(in.graw[v], g);
      unpack_codes<EFM>(in.cw, v, c);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float sc = c[e] * u;
        const float d = sc + lo;
        a[v][e] = g[e] + d;
      }
    }
  }
  if (!full) {  // elements past the end of the tensor are 0 and never kept
    const int r = opaque_v(rem);
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (8 * v + e >= r) a[v][e] = 0.0f;
  }
}

// ------------------------------------------- buckets spanning Top-K blocks
// With buckets of B_q >= B_d elements (Section 3.1 mentions B_q = 100K) a
// bucket holds several blocks and a block may straddle two buckets.  The
// (delta, Delta) pairs of a tensor's buckets live in two tables: step t
// decodes with table (t-1) mod 2 and fills table t mod 2.  The select kernel
// then writes, per block, the (min, max) of the residual in each of its (at
// most two) buckets; a reduction turns them into the new table, and a second
// pass over the block quantizes the residual with it.

// The lane's two buckets: its elements [0, sp) lie in the first, the rest
// in the next.  `table`: the pairs of step t's decode (0) or of step t (1).
struct LqBuckets {
  u32x2 st[2];
  int sp;
};

__device__ __forceinline__ LqBuckets lq_buckets(const StepParams& p, const Block& b, uint32_t eb, int epl,
                                                int table) {
  const int64_t bq = p.big_bucket;
  const int64_t el = b.e0 + eb;  // tensor element of the lane's first element
  const int64_t bk = el / bq;
  const int64_t sp = (bk + 1) * bq - el;
  const uint64_t t = (uint64_t)((p.t - 1 + table) & 1);
  const Rsrc rt = make_rsrc(p.state + p.stats_plane + t * p.table_bytes + (uint64_t)b.desc.first_bucket * 8,
                            (uint32_t)(b.desc.num_buckets * 8));
  LqBuckets r;
  r.st[0] = __builtin_amdgcn_raw_buffer_load_b64(rt, (uint32_t)(bk * 8), 0, 0);
  r.st[1] = __builtin_amdgcn_raw_buffer_load_b64(rt, (uint32_t)(bk * 8 + 8), 0, 0);  // past the end: 0
  r.sp = sp < epl ? (int)sp : epl;
  return r;
}

// a = g + Q^-1(e) with the lane's two buckets (the arithmetic of lane_decode).
template <int EPL, bool GBF16, int EFM>
__device__ __forceinline__ void lane_decode_lq(const LaneIn<EPL, true, GBF16, EFM>& in, const LqBuckets& bk,
                                               float (&a)[EPL / 8][8], int rem, bool full) {
  constexpr int NV = EPL / 8;
  const float lo0 = __uint_as_float(bk.st[0][0]), u0 = ef_step<EFM>(__uint_as_float(bk.st[0][1]) - lo0);
  const float lo1 = __uint_as_float(bk.st[1][0]), u1 = ef_step<EFM>(__uint_as_float(bk.st[1][1]) - lo1);
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    float g[8], c[8];
    unpack8<GBF16>(in.graw[v], g);
    unpack_codes<EFM>(in.cw, v, c);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const bool second = 8 * v + e >= bk.sp;
      const float lo = second ? lo1 : lo0, u = second ? u1 : u0;
      const float sc = c[e] * u;
      const float d = sc + lo;
      a[v][e] = g[e] + d;
    }
  }
  if (!full) {
    const int r = opaque_v(rem);
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (8 * v + e >= r) a[v][e] = 0.0f;
  }
}

template <int EPL>
__device__ __forceinline__ void lane_vmax(const float (&a)[EPL / 8][8], float (&vmax)[EPL / 8]) {
#pragma unroll
  for (int v = 0; v < EPL / 8; ++v) {
    const float m0 = __builtin_fmaxf(__builtin_fmaxf(__builtin_fabsf(a[v][0]), __builtin_fabsf(a[v][1])), __builtin_fabsf(a[v][2]));
    const float m1 = __builtin_fmaxf(__builtin_fmaxf(m0, __builtin_fabsf(a[v][3])), __builtin_fabsf(a[v][4]));
    const float m2 = __builtin_fmaxf(__builtin_fmaxf(m1, __builtin_fabsf(a[v][5])), __builtin_fabsf(a[v][6]));
    vmax[v] = __builtin_fmaxf(m2, __builtin_fabsf(a[v][7]));
  }
}

// Where the randomized quantizer's xi come from: element i of tensor j at
// step t takes word i mod 4 of Philox4x32-10 at counter (i/4 low, i/4 high,
// j, t) under the 64-bit seed, and xi = (word >> 8) * 2^-24.
struct EfStream {
  int64_t e0;      // first element of the block in its tensor
  uint32_t j, t;   // tensor number, step
  uint32_t k0, k1; // seed, low and high word
};

// The 24-bit integers w of xi = w * 2^-24 for the 8 elements starting at
// tensor element 4*quad (two Philox blocks).
__device__ __forceinline__ void philox_w24(uint64_t quad, const EfStream& st, uint32_t (&w24)[8]) {
#pragma unroll
  for (int h = 0; h < 2; ++h) {
    const uint64_t qh = quad + h;
    const u32x4 r = philox4x32_10(u32x4{(uint32_t)qh, (uint32_t)(qh >> 32), st.j, st.t}, st.k0, st.k1);
#pragma unroll
    for (int i = 0; i < 4; ++i) w24[4 * h + i] = r[i] >> 8;
  }
}

// Codes of one vector of 8 elements x against one bucket (lower bound mnv,
// quantization step uv): 4-bit codes in w[0], element e in bits [4e, 4e + 4);
// 8-bit codes in w[0], w[1], element e in byte e & 3 of word e / 4.  quad:
// the tensor element number of x[0], divided by 4 (the randomized rounding's
// counter).
template <int EFM>
__device__ __forceinline__ void vector_codes(const float (&x)[8], float mnv, float uv, uint64_t quad,
                                             const EfStream& st, uint32_t (&w)[(EFM & kEf8) ? 2 : 1]) {
  constexpr bool EF8 = (EFM & kEf8) != 0;
  constexpr int CW = EF8 ? 2 : 1;
  constexpr float L = EF8 ? 255.0f : 15.0f;
  if constexpr ((EFM & kEfRandom) != 0) {
    // the vector starts at a multiple of 8 within the tensor
    uint32_t w24[8];
    philox_w24(quad, st, w24);
#pragma unroll
    for (int c = 0; c < CW; ++c) w[c] = 0;
    if (uv != 0.0f) {
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const uint32_t code = code_randomized(x[e], mnv, uv, L, w24[e]);
        if constexpr (EF8) w[e >> 2] |= code << (8 * (e & 3));
        else w[0] |= code << (4 * e);
      }
    }
  } else {
    // Codes from two products that bracket the quotient: v_rcp is within
    // 1 ulp for these u, so r_lo < 1/u < r_hi and
    // rint((x-min)*r_lo) <= rint((x-min)/u) <= rint((x-min)*r_hi).  Where
    // the two agree (all but a few elements in a million) the code is
    // exact; elsewhere it is recomputed with an IEEE division.
    const float rcp = __builtin_amdgcn_rcpf(uv);
    const float r_lo = __uint_as_float(__float_as_uint(rcp) - 2u);
    const float r_hi = __uint_as_float(__float_as_uint(rcp) + 2u);
    bool agree;
    if constexpr (EF8) {
      uint32_t d1a = 0, d1b = 0, d2a = 0, d2b = 0;
#pragma unroll
      for (int h = 0; h < 4; ++h) {
        const float ya = x[h] - mnv, yb = x[4 + h] - mnv;
        d1a = __builtin_amdgcn_cvt_pk_u8_f32(ya * r_lo, h, d1a);  // round half to even, clamp to [0, 255]
        d1b = __builtin_amdgcn_cvt_pk_u8_f32(yb * r_lo, h, d1b);
        d2a = __builtin_amdgcn_cvt_pk_u8_f32(ya * r_hi, h, d2a);
        d2b = __builtin_amdgcn_cvt_pk_u8_f32(yb * r_hi, h, d2b);
      }
      w[0] = d1a;
      w[CW - 1] = d1b;
      agree = (d1a == d2a) & (d1b == d2b);
    } else {
      uint32_t d1e = 0, d1o = 0, d2e = 0, d2o = 0;
#pragma unroll
      for (int h = 0; h < 4; ++h) {
        const float ye = x[2 * h] - mnv, yo = x[2 * h + 1] - mnv;
        const float p1e = ye * r_lo, p1o = yo * r_lo;
        const float p2e = ye * r_hi, p2o = yo * r_hi;
        d1e = __builtin_amdgcn_cvt_pk_u8_f32(p1e, h, d1e);  // round half to even, clamp to [0, 255]
        d1o = __builtin_amdgcn_cvt_pk_u8_f32(p1o, h, d1o);
        d2e = __builtin_amdgcn_cvt_pk_u8_f32(p2e, h, d2e);
        d2o = __builtin_amdgcn_cvt_pk_u8_f32(p2o, h, d2o);
      }
      w[0] = d1e | (d1o << 4);
      agree = (d1e == d2e) & (d1o == d2o);
    }
    const bool exact_u = uv >= 0x1p-125f && uv <= 0x1p+125f;
    if (!exact_u | !agree) {
#pragma unroll
      for (int c = 0; c < CW; ++c) w[c] = 0;
      if (uv != 0.0f) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float y = x[e] - mnv;
          float rr = __builtin_rintf(y / uv);
          rr = __builtin_fminf(__builtin_fmaxf(rr, 0.0f), L);
          if constexpr (EF8) w[e >> 2] |= (uint32_t)rr << (8 * (e & 3));
          else w[0] |= (uint32_t)rr << (4 * e);
        }
      }
    }
  }
}

// Stores a lane's codes (the layout of vector_codes, vector after vector).
// `wide`: 16-byte accesses for 4-bit codes (the block fills every lane of the
// kernel); 8-bit codes always take them, since B_d is a multiple of 16 and an
// access then lies wholly inside or wholly past the block's codes.
template <int EPL, int EFM>
__device__ __forceinline__ void lane_store_codes(const uint32_t (&wv)[(EPL / 8) * ((EFM & kEf8) ? 2 : 1)],
                                                 uint32_t eb, bool wide, Rsrc re) {
  constexpr int NV = EPL / 8;
  if constexpr ((EFM & kEf8) != 0) {
#pragma unroll
    for (int q = 0; q < NV / 2; ++q)
      __builtin_amdgcn_raw_buffer_store_b128(u32x4{wv[4 * q], wv[4 * q + 1], wv[4 * q + 2], wv[4 * q + 3]}, re,
                                             eb + 16 * q, 0, 0);
  } else if (NV > 2 && wide) {
#pragma unroll
    for (int q = 0; q < NV / 4; ++q)
      __builtin_amdgcn_raw_buffer_store_b128(u32x4{wv[4 * q], wv[4 * q + 1], wv[4 * q + 2], wv[4 * q + 3]}, re,
                                             (eb >> 1) + 16 * q, 0, 0);
  } else {
#pragma unroll
    for (int q = 0; q < NV / 2; ++q)
      __builtin_amdgcn_raw_buffer_store_b64(u32x2{wv[2 * q], wv[2 * q + 1]}, re, (eb >> 1) + 8 * q, 0, 0);
  }
}

// ------------------------------------- coalesced block loads and stores
// One wave over a 4096-element block (64 elements per lane: lane l owns
// [64l, 64l + 64)) with bf16 gradients.  A lane's own run is 128 bytes of
// gradient and 32 (4-bit) or 64 (8-bit) bytes of codes, so loading it
// directly gives every 16-byte access of the wave a 128-byte (or 32- or
// 64-byte) stride.  Instead
// the wave loads the block as contiguous kilobytes (access v of lane l is
// bytes 1024v + 16l) with the nt policy, and the data reaches its owner
// through LDS.  Layouts in LDS (byte offsets; the padding keeps 16 lanes'
// 16-byte reads on distinct banks):
//   gradient: element e of a half block at 2e + 16*(e / 64), 4608 bytes per
//     half (a half is 32 lanes' runs, loaded by accesses 0-3 or 4-7);
//   4-bit codes: code byte c at kTrCodes + c + 16*(c / 32), 3072 bytes;
//   8-bit codes: code byte c at c + 16*(c / 64), 5120 bytes, exchanged
//     before the gradient through the start of the same LDS.
// The two halves of the gradient pass one after the other through the same
// 4608 bytes, so the exchange needs 7680 bytes of LDS.
constexpr uint32_t kTrCodes = 4608;
constexpr uint32_t kTrBytes = 7680;
constexpr uint32_t kTrCodes8Bytes = 5120;
static_assert(kTrBytes <= select_lds_words() * 4, "the exchange reuses the select kernel's LDS");
static_assert(kTrCodes8Bytes <= kTrBytes, "the 8-bit code exchange fits the same LDS");

struct CoalescedIn {
  u32x4 g[8];
  u32x4 c[4];  // codes: 2 accesses (4-bit) or 4 (8-bit)
};

template <int EFM>
__device__ __forceinline__ void coalesced_load_codes(CoalescedIn& x, Rsrc re, int lane) {
#pragma unroll
  for (int q = 0; q < ((EFM & kEf8) ? 4 : 2); ++q)
    x.c[q] = __builtin_amdgcn_raw_buffer_load_b128(re, 1024 * q + 16 * lane, 0, kStream);
}
__device__ __forceinline__ void coalesced_load_grad(CoalescedIn& x, Rsrc rg, int lane) {
#pragma unroll
  for (int v = 0; v < 8; ++v) x.g[v] = __builtin_amdgcn_raw_buffer_load_b128(rg, 1024 * v + 16 * lane, 0, kStream);
}

// Hands the loaded block to the lanes that own it: lane l's gradient vectors
// (8 elements each) and code words (8 codes each) in element order.
template <bool LB, int EFM>
__device__ __forceinline__ void coalesced_exchange(const CoalescedIn& x, LaneIn<64, LB, true, EFM>& in,
                                                   uint32_t* lds, int lane) {
  constexpr bool EF8 = (EFM & kEf8) != 0;
  uint8_t* const b = (uint8_t*)lds;
  const uint32_t wg = 16u * (uint32_t)lane + 16u * (uint32_t)(lane >> 3);  // + 1152v: access v of this lane
  const uint32_t rg = 144u * (uint32_t)(lane & 31);                         // + 16V: this lane's vector V
  if constexpr (EF8) {
    // access q of lane l holds lane 16q + l/4's bytes 16*(l mod 4) ...
#pragma unroll
    for (int q = 0; q < 4; ++q) *(u32x4*)(b + 1280 * q + 80 * (lane >> 2) + 16 * (lane & 3)) = x.c[q];
    wave_sync();
#pragma unroll
    for (int h = 0; h < 4; ++h) {
      const u32x4 t = *(const u32x4*)(b + 80 * lane + 16 * h);
#pragma unroll
      for (int j = 0; j < 4; ++j) in.cw[4 * h + j] = t[j];
    }
    wave_sync();
  }
#pragma unroll
  for (int v = 0; v < 4; ++v) *(u32x4*)(b + 1152 * v + wg) = x.g[v];
  if constexpr (!EF8) {
#pragma unroll
    for (int q = 0; q < 2; ++q)
      *(u32x4*)(b + kTrCodes + 1536 * q + 16 * lane + 16 * (lane >> 1)) = x.c[q];
  }
  wave_sync();
  if (lane < 32) {
#pragma unroll
    for (int v = 0; v < 8; ++v) in.graw[v].w[0] = *(const u32x4*)(b + rg + 16 * v);
  }
  if constexpr (!EF8) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const u32x4 t = *(const u32x4*)(b + kTrCodes + 48 * lane + 16 * h);
#pragma unroll
      for (int j = 0; j < 4; ++j) in.cw[4 * h + j] = t[j];
    }
  }
  wave_sync();
#pragma unroll
  for (int v = 0; v < 4; ++v) *(u32x4*)(b + 1152 * v + wg) = x.g[4 + v];
  wave_sync();
  if (lane >= 32) {
#pragma unroll
    for (int v = 0; v < 8; ++v) in.graw[v].w[0] = *(const u32x4*)(b + rg + 16 * v);
  }
  wave_sync();
}

// Stores the lane's codes (4-bit: one word per vector; 8-bit: two) through
// LDS as coalesced 16-byte accesses with the nt policy, in the layouts of the
// exchange; the whole record of the block is written (codes past the block's
// end are 0).
template <int EFM>
__device__ __forceinline__ void lane_store_codes_coalesced(const uint32_t (&wv)[(EFM & kEf8) ? 16 : 8],
                                                           uint32_t* lds, Rsrc re) {
  const int lane = thread_id() & (kWave - 1);
  wave_sync();
  if constexpr ((EFM & kEf8) != 0) {
    uint8_t* const b = (uint8_t*)lds;
#pragma unroll
    for (int h = 0; h < 4; ++h)
      *(u32x4*)(b + 80 * lane + 16 * h) = u32x4{wv[4 * h], wv[4 * h + 1], wv[4 * h + 2], wv[4 * h + 3]};
    wave_sync();
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const u32x4 t = *(const u32x4*)(b + 1280 * q + 80 * (lane >> 2) + 16 * (lane & 3));
      __builtin_amdgcn_raw_buffer_store_b128(t, re, 1024 * q + 16 * lane, 0, kStream);
    }
  } else {
    uint8_t* const b = (uint8_t*)lds + kTrCodes;
#pragma unroll
    for (int h = 0; h < 2; ++h)
      *(u32x4*)(b + 48 * lane + 16 * h) = u32x4{wv[4 * h], wv[4 * h + 1], wv[4 * h + 2], wv[4 * h + 3]};
    wave_sync();
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const u32x4 t = *(const u32x4*)(b + 1536 * q + 16 * lane + 16 * (lane >> 1));
      __builtin_amdgcn_raw_buffer_store_b128(t, re, 1024 * q + 16 * lane, 0, kStream);
    }
  }
}

// a[I] = 0 (Algorithm 1): the kept elements are |a| > T, and |a| == T up to
// index i_last; every |a| >= T when notie.
template <int EPL>
__device__ __forceinline__ void lane_zero_kept(float (&a)[EPL / 8][8], uint32_t T, bool notie, uint32_t i_last,
                                               uint32_t eb) {
  constexpr int NV = EPL / 8;
  // kept elements: |a| > T, and |a| == T up to index i_last; without ties
  // at the threshold that is |a| >= T (a wave-uniform case).  With ties the
  // kept elements equal to T are zeroed first, and the rest are those
  // with |a| >= the next float above T.
  uint32_t Tk = T;
  if (!notie) {
    const float tf = opaque_f(__uint_as_float(T));
    const int last_here = (int)i_last - (int)eb;  // this lane's elements up to i_last: [0, last_here]
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if ((__builtin_fabsf(a[v][e]) == tf) & (8 * v + e <= last_here)) a[v][e] = 0.0f;
    Tk = T + 1u;
  }
  // (the values pass through an empty asm so that the compiler does not
  // carry |a| of the tie pass into the test below in extra registers)
#pragma unroll
  for (int v = 0; v < NV; ++v)
#pragma unroll
    for (int e = 0; e < 8; ++e) asm volatile("" : "+v"(a[v][e]));
  {
    const float tk = __uint_as_float(Tk);
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
      for (int e = 0; e < 8; ++e) a[v][e] = (__builtin_fabsf(a[v][e]) >= tk) ? 0.0f : a[v][e];
  }
}

// e = Q(a with a[I] = 0) (Algorithm 1; Algorithm 2, Q; Section 3.1; with
// kEfRandom the randomized Q of Lemma 1): zeroes the kept elements (|a| >
// T, and |a| == T up to index i_last; every |a| >= T when notie), computes
// the bucket (min, max) pairs and the codes, and stores both.
// KEPT_ZEROED: the caller has zeroed the kept elements already.
//
// tr_lds (one-wave kernels with 64 elements per lane, over a whole-lane
// block): the codes leave through LDS as coalesced 16-byte stores
// (lane_store_codes_coalesced), and the bucket pairs with the nt policy.
template <int EPL, bool LB, int EFM = 0, bool KEPT_ZEROED = false>
__device__ __forceinline__ void lane_quantize_store(float (&a)[EPL / 8][8], uint32_t T, bool notie,
                                                    uint32_t i_last, uint32_t eb, int s, int rem, bool full, int bl,
                                                    bool wide, Rsrc re, Rsrc rs, const EfStream& rs_ef = {},
                                                    uint32_t* tr_lds = nullptr) {
  constexpr int NV = EPL / 8;
  constexpr bool EF8 = (EFM & kEf8) != 0;
  constexpr int CW = EF8 ? 2 : 1;
  constexpr int lg = EPL == 16 ? 4 : EPL == 32 ? 5 : 6;
  if constexpr (!KEPT_ZEROED) lane_zero_kept<EPL>(a, T, notie, i_last, eb);
  // bucket min / max: per vector, then over the vectors of a bucket inside
  // the lane, then over the lanes of a bucket
  float mn[NV], mx[NV];
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    if (full) {
      mn[v] = __builtin_fminf(__builtin_fminf(__builtin_fminf(a[v][0], a[v][1]), a[v][2]),
                              __builtin_fminf(__builtin_fminf(a[v][3], a[v][4]), a[v][5]));
      mn[v] = __builtin_fminf(mn[v], __builtin_fminf(a[v][6], a[v][7]));
      mx[v] = __builtin_fmaxf(__builtin_fmaxf(__builtin_fmaxf(a[v][0], a[v][1]), a[v][2]),
                              __builtin_fmaxf(__builtin_fmaxf(a[v][3], a[v][4]), a[v][5]));
      mx[v] = __builtin_fmaxf(mx[v], __builtin_fmaxf(a[v][6], a[v][7]));
    } else {
      mn[v] = __builtin_inff();
      mx[v] = -__builtin_inff();
      const int r = opaque_v(rem);
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (8 * v + e < r) { mn[v] = __builtin_fminf(mn[v], a[v][e]); mx[v] = __builtin_fmaxf(mx[v], a[v][e]); }
    }
  }
  if constexpr (LB) {
    float lo = mn[0], hi = mx[0];
#pragma unroll
    for (int v = 1; v < NV; ++v) {
      lo = __builtin_fminf(lo, mn[v]);
      hi = __builtin_fmaxf(hi, mx[v]);
    }
    group_minmax(lo, hi, bl - lg);
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      mn[v] = lo;
      mx[v] = hi;
    }
  } else {
    // B_q = 8 << j vectors... combine the 2^j vectors of each bucket
#pragma unroll
    for (int j = 0; (1 << j) < NV; ++j) {
      if (bl - 3 > j) {
#pragma unroll
        for (int v = 0; v < NV; ++v) {
          const int w = v ^ (1 << j);
          if (w > v) {
            const float l2 = __builtin_fminf(mn[v], mn[w]), h2 = __builtin_fmaxf(mx[v], mx[w]);
            mn[v] = mn[w] = l2;
            mx[v] = mx[w] = h2;
          }
        }
      }
    }
  }
  uint32_t wv[NV * CW];
  {
    float uq = 0.0f, mnq = 0.0f;
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      if (!LB || v == 0) {
        mn[v] = mn[v] + 0.0f;  // a bucket bound of -0 is stored as +0
        mx[v] = mx[v] + 0.0f;
        mnq = mn[v];
        uq = ef_step<EFM>(mx[v] - mn[v]);
      }
      const float uv = uq, mnv = mnq;
      uint32_t w[CW];
      vector_codes<EFM>(a[v], mnv, uv, (uint64_t)(rs_ef.e0 + eb + 8 * v) >> 2, rs_ef, w);
      if (!full) {
        const int r = opaque_v(rem);
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if (8 * v + e >= r) {
            if constexpr (EF8) w[e >> 2] &= ~(0xFFu << (8 * (e & 3)));
            else w[0] &= ~(0xFu << (4 * e));
          }
      }
#pragma unroll
      for (int c = 0; c < CW; ++c) wv[CW * v + c] = w[c];
    }
  }
  if constexpr (EPL == 64) {
    if (tr_lds != nullptr) {
      // every lane takes part in the exchange; codes past s are 0
      lane_store_codes_coalesced<EFM>(wv, tr_lds, re);
      if constexpr (LB) {
        if ((int)eb < s && (eb & ((1u << bl) - 1)) == 0)
          __builtin_amdgcn_raw_buffer_store_b64(u32x2{__float_as_uint(mn[0]), __float_as_uint(mx[0])}, rs,
                                                (eb >> bl) * 8, 0, kStream);
        return;
      }
    }
  }
  if ((int)eb < s) {
    if (tr_lds == nullptr) lane_store_codes<EPL, EFM>(wv, eb, wide, re);
    if constexpr (LB) {
      if ((eb & ((1u << bl) - 1)) == 0)
        __builtin_amdgcn_raw_buffer_store_b64(u32x2{__float_as_uint(mn[0]), __float_as_uint(mx[0])}, rs,
                                              (eb >> bl) * 8, 0, 0);
    } else {
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        const uint32_t e0 = eb + 8 * v;
        if ((e0 & ((1u << bl) - 1)) == 0 && (int)e0 < s)
          __builtin_amdgcn_raw_buffer_store_b64(u32x2{__float_as_uint(mn[v]), __float_as_uint(mx[v])}, rs,
                                                (e0 >> bl) * 8, 0, 0);
      }
    }
  }
}

// The (min, max) of the residual of the wave's elements in the block's first
// bucket and in the next one (elements past the block's end excluded; an
// empty part gives (+inf, -inf)), reduced over the wave: out = (min0, max0,
// min1, max1) in every lane.
template <int EPL>
__device__ __forceinline__ void wave_partials(const float (&a)[EPL / 8][8], const StepParams& p, const Block& b,
                                              uint32_t eb, int rem, float (&out)[4]) {
  constexpr int NV = EPL / 8;
  const int64_t bq = p.big_bucket;
  const int64_t split = ((b.e0 / bq) + 1) * bq - b.e0;  // block element where the next bucket starts
  const int64_t ls = split - (int64_t)eb;
  const int lsplit = ls < 0 ? 0 : ls > EPL ? EPL : (int)ls;
  const int r = opaque_v(rem);
  float mn0 = __builtin_inff(), mx0 = -__builtin_inff(), mn1 = __builtin_inff(), mx1 = -__builtin_inff();
#pragma unroll
  for (int v = 0; v < NV; ++v)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int i = 8 * v + e;
      const float x = a[v][e];
      if (i < r) {
        if (i < lsplit) {
          mn0 = __builtin_fminf(mn0, x);
          mx0 = __builtin_fmaxf(mx0, x);
        } else {
          mn1 = __builtin_fminf(mn1, x);
          mx1 = __builtin_fmaxf(mx1, x);
        }
      }
    }
#pragma unroll
  for (int d = 1; d < kWave; d <<= 1) {
    mn0 = __builtin_fminf(mn0, __shfl_xor(mn0, d, kWave));
    mx0 = __builtin_fmaxf(mx0, __shfl_xor(mx0, d, kWave));
    mn1 = __builtin_fminf(mn1, __shfl_xor(mn1, d, kWave));
    mx1 = __builtin_fmaxf(mx1, __shfl_xor(mx1, d, kWave));
  }
  out[0] = mn0;
  out[1] = mx0;
  out[2] = mn1;
  out[3] = mx1;
}

// A block's partials (its first bucket's and the next one's (min, max))
// to the partials plane.
__device__ __forceinline__ void store_partials(const StepParams& p, int64_t gb, const float (&x)[4]) {
  const Rsrc rp = make_rsrc(p.state + p.partial_plane + (uint64_t)gb * 16, 16);
  __builtin_amdgcn_raw_buffer_store_b128(
      u32x4{__float_as_uint(x[0]), __float_as_uint(x[1]), __float_as_uint(x[2]), __float_as_uint(x[3])}, rp, 0, 0, 0);
}

// Per block and bucket, the (min, max) of the residual for a block held by
// one wave: the wave's partials, written by lane 0.
template <int EPL>
__device__ __forceinline__ void lane_partials(const float (&a)[EPL / 8][8], const StepParams& p, const Block& b,
                                              uint32_t eb, int rem, int64_t gb) {
  float x[4];
  wave_partials<EPL>(a, p, b, eb, rem, x);
  if (thread_id() == 0) store_partials(p, gb, x);
}

// Blocks above this size take the multi-wave select and the per-quarter
// update; their window records carry a table of segment starts per quarter
// of kQuarter elements.
constexpr int kSubBlock = 4096;
constexpr int kQuarter = 1024;

}  // namespace
}  // namespace microadam
