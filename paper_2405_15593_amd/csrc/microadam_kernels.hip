// MicroAdam step kernels for CDNA4 (gfx950).
//
// One optimizer step is two launches over all Top-K blocks (B_d elements of
// one tensor each; blocks share nothing):
//
//   select_kernel   one wave per block (lane l: elements [l*EPL, (l+1)*EPL)):
//     1. a = g + Q^-1(e)                          (Algorithm 1; Algorithm 2, Q^-1)
//     2. block Top-K of |a|, lower index wins ties (Section 3.1, "Top-K")
//     3. the new window row (I, bf16(V)) is stored (Section 3.2)
//     4. a[I] = 0; bucket (delta, Delta) = (min, max) in the lane or by lane
//        shuffles; e = Q(a, delta, Delta), two 4-bit codes per byte
//        (Algorithm 1; Section 3.1)
//
//   update_kernel   one workgroup of 256 threads per block (thread tid: the
//   16 consecutive elements tid*16 + [0, 16) of the block):
//     5. one wave rebuilds m-hat, v-hat of the block's window entries in LDS
//        from the m rows with weights beta^(t-s) (Algorithm 2, AdamStats)
//     6. every wave applies theta <- (1 - eta*lambda) theta
//        - eta m / (eps + sqrt(v)) to its elements (Algorithm 1; Algorithm 4)
//
// Splitting the step costs one extra read of the new window row (4 bytes per
// kept entry) and lets each kernel keep a small register and LDS footprint.
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
  // the entry with its index replaced by w (an accumulator word, < 2^16)
  __device__ static T with_word(T e, uint32_t w) {
    if constexpr (VF32) return u32x2{w, e[1]};
    else return (e & 0xFFFF0000u) | w;
  }
  __device__ static uint32_t word(T e) {
    if constexpr (VF32) return e[0];
    else return e & 0xFFFFu;
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
  uint32_t j;             // tensor number
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
template <int EPL, bool LB, int EFM = 0>
__device__ __forceinline__ void lane_quantize_store(float (&a)[EPL / 8][8], uint32_t T, bool notie,
                                                    uint32_t i_last, uint32_t eb, int s, int rem, bool full, int bl,
                                                    bool wide, Rsrc re, Rsrc rs, const EfStream& rs_ef = {}) {
  constexpr int NV = EPL / 8;
  constexpr bool EF8 = (EFM & kEf8) != 0;
  constexpr int CW = EF8 ? 2 : 1;
  constexpr int lg = EPL == 16 ? 4 : EPL == 32 ? 5 : 6;
  lane_zero_kept<EPL>(a, T, notie, i_last, eb);
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
  if ((int)eb < s) {
    lane_store_codes<EPL, EFM>(wv, eb, wide, re);
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

// Per block and bucket, the (min, max) of the residual (elements past the
// block's end excluded; an empty part gives (+inf, -inf)): pairs for the
// block's first bucket and for the next one, written by lane 0.
template <int EPL>
__device__ __forceinline__ void lane_partials(const float (&a)[EPL / 8][8], const StepParams& p, const Block& b,
                                              uint32_t eb, int rem, int64_t gb) {
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
  if (thread_id() == 0) {
    const Rsrc rp = make_rsrc(p.state + p.partial_plane + (uint64_t)gb * 16, 16);
    __builtin_amdgcn_raw_buffer_store_b128(
        u32x4{__float_as_uint(mn0), __float_as_uint(mx0), __float_as_uint(mn1), __float_as_uint(mx1)}, rp, 0, 0, 0);
  }
}

template <int EPL, bool LB, bool GBF16, bool VF32, int EFM, bool LQ = false>
__global__ void __launch_bounds__(kWave) __attribute__((amdgpu_waves_per_eu(4)))
select_kernel(StepParams p, int64_t first) {
  static_assert(!LQ || (EPL == 64 && LB && (EFM & kEfRandom) == 0), "buckets spanning blocks: 64 per lane");
  constexpr int NV = EPL / 8;
  constexpr int CAP = kWave * EPL;
  using E = Entry<VF32>;
  extern __shared__ __align__(16) uint32_t smem[];
  float* const regv = (float*)smem;                  // [kMaxCandVec][8] candidate vectors
  uint32_t* const regi = smem + kMaxCandVec * 8;     // [kMaxCandVec] their first element
  float* const cval = (float*)(regi + kMaxCandVec);  // [kCandMax] candidate values
  uint32_t* const cidx = (uint32_t*)(cval + kCandMax);  // [kCandMax] candidate indices
  uint32_t* const rowbuf = cidx + kCandMax;          // [kRowBufWords] the new row's lines

  const int lane = thread_id();
  const uint32_t eb = (uint32_t)lane * EPL;  // first element of this lane
  const int bl = p.bucket_log2;
  const int64_t gb = first + block_id();

  // The block's EF codes and bucket pairs are addressed by gb alone, so their
  // loads go out before the tensor lookup that the gradient needs.
  const uint32_t nbk = (uint32_t)(p.block >> bl);
  const uint32_t ef_bytes = (EFM & kEf8) ? (uint32_t)p.block : (uint32_t)(p.block >> 1);
  const Rsrc re = make_rsrc(p.state + p.ef_plane + (uint64_t)gb * ef_bytes, ef_bytes);
  const Rsrc rs = make_rsrc(p.state + p.stats_plane + (uint64_t)gb * nbk * 8, nbk * 8);
  const bool wide = p.block == CAP;
  LaneIn<EPL, LB, GBF16, EFM> in;
  if constexpr (LQ) lane_load_codes(in, re, eb, wide);
  else lane_load_state(in, re, rs, eb, bl, wide);
  const Block b = locate(p, gb);
  LqBuckets lqb = {};
  if constexpr (LQ) lqb = lq_buckets(p, b, eb, EPL, 0);
  const int s = b.s, kq = b.kq;
  const bool full = s == CAP;
  const Rsrc rg = make_rsrc((const uint8_t*)b.desc.grad + b.e0 * (GBF16 ? 2 : 4), vec_bytes<GBF16>(s));
  lane_load_grad(in, rg, eb);
  // The new row, bytes [row_lo, row_hi) of the block's window record, is
  // written as the whole 128-byte lines [span_lo, span_hi) that cover it
  // (records are whole lines): partial-line writes cost the memory system
  // far more than their bytes.  The words of the first and last line that
  // lie outside the row are read here and written back unchanged.
  constexpr uint32_t EB = VF32 ? 8u : 4u;
  const uint32_t row_lo = (uint32_t)p.new_slot * (uint32_t)kq * EB;
  const uint32_t row_hi = row_lo + (uint32_t)kq * EB;
  const uint32_t span_lo = row_lo & ~127u, span_hi = (row_hi + 127u) & ~127u;
  const Rsrc rrec = make_rsrc(p.state + p.win_plane + (uint64_t)gb * p.win_stride, (uint32_t)p.win_stride);
  const uint32_t edge_off = lane < 32 ? span_lo + 4 * lane : span_hi - 128 + 4 * (lane - 32);
  const uint32_t edge_old = __builtin_amdgcn_raw_buffer_load_b32(rrec, edge_off, 0, 0);

  // ---------------------------------------------- 1. a = g + Q^-1(e)
  float a[NV][8];
  const int rem = s - (int)eb;  // this lane's elements below the end of the block: [0, rem)
  if constexpr (LQ) lane_decode_lq(in, lqb, a, rem, full);
  else lane_decode(in, a, rem, full);

  // ---------------------------------------------- 2. Top-K threshold
  float vmax[NV];
  lane_vmax<EPL>(a, vmax);
  const Rsrc rw = window_rsrc<VF32 ? 2 : 1>(p, gb, kq);
  const uint32_t row0 = (uint32_t)p.new_slot * kq;

  uint32_t T = 0, i_last = 0;
  bool notie = false;
  bool general = kq > 2 * kWave;
  if (!general) {
    // stage 1: L over the half-lane maxima
    float h0 = vmax[0], h1 = vmax[NV / 2];
#pragma unroll
    for (int v = 1; v < NV / 2; ++v) {
      h0 = __builtin_fmaxf(h0, vmax[v]);
      h1 = __builtin_fmaxf(h1, vmax[NV / 2 + v]);
    }
    const uint32_t hb0 = __float_as_uint(h0), hb1 = __float_as_uint(h1);
    uint32_t P = 0;
#pragma unroll
    for (int bit = 30; bit >= 18; --bit) {
      const uint32_t c = P | (1u << bit);
      if ((int)(popc(ballot(hb0 >= c)) + popc(ballot(hb1 >= c))) >= kq) P = c;
    }
    const uint32_t Lb = P;
    const float L = __uint_as_float(Lb);

    // stage 2a: candidate vectors to LDS, in element order
    bool f[NV];
    uint32_t cnt = 0;
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      f[v] = vmax[v] >= L;
      cnt += f[v] ? 1u : 0u;
    }
    uint32_t nvec;
    const uint32_t pre = lane_prefix(cnt, nvec);
    general = Lb == 0 || nvec > (uint32_t)kMaxCandVec;
    if (!general) {
      {
        uint32_t pos = pre;
#pragma unroll
        for (int v = 0; v < NV; ++v) {
          if (f[v]) {
            *(float4*)(regv + pos * 8) = make_float4(a[v][0], a[v][1], a[v][2], a[v][3]);
            *(float4*)(regv + pos * 8 + 4) = make_float4(a[v][4], a[v][5], a[v][6], a[v][7]);
            regi[pos] = eb + 8 * v;
            ++pos;
          }
        }
      }
      wave_sync();
      // stage 2b: elements >= L of candidate vectors lane and lane + 64
      uint32_t C = 0;
      auto gather = [&](auto nsv_tag) {
        constexpr int NSV = decltype(nsv_tag)::value;
        float cv[NSV][8];
        uint32_t cb[NSV], base[NSV], cc[NSV];
        uint32_t total = 0;
#pragma unroll
        for (int r = 0; r < NSV; ++r) {
          const uint32_t j = lane + kWave * r;
          const bool have = j < nvec;
          const uint32_t src = have ? j : 0u;
          const float4 x0 = *(const float4*)(regv + src * 8);
          const float4 x1 = *(const float4*)(regv + src * 8 + 4);
          cb[r] = regi[src];
          cv[r][0] = x0.x; cv[r][1] = x0.y; cv[r][2] = x0.z; cv[r][3] = x0.w;
          cv[r][4] = x1.x; cv[r][5] = x1.y; cv[r][6] = x1.z; cv[r][7] = x1.w;
          uint32_t c = 0;
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            if (!have) cv[r][e] = 0.0f;  // key 0 < L: never a candidate
            c += __builtin_fabsf(cv[r][e]) >= L ? 1u : 0u;
          }
          cc[r] = c;
        }
#pragma unroll
        for (int r = 0; r < NSV; ++r) {
          uint32_t t;
          base[r] = total + lane_prefix(cc[r], t);
          total += t;
        }
        C = total;
        if (C <= (uint32_t)kCandMax) {
#pragma unroll
          for (int r = 0; r < NSV; ++r) {
            uint32_t pos = base[r];
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              if (__builtin_fabsf(cv[r][e]) >= L) {
                cval[pos] = cv[r][e];
                cidx[pos] = cb[r] + e;
                ++pos;
              }
            }
          }
        }
      };
      if (nvec <= (uint32_t)kWave) gather(std::integral_constant<int, 1>{});
      else gather(std::integral_constant<int, 2>{});
      general = C > (uint32_t)kCandMax || C < (uint32_t)kq;
      if (!general) {
        wave_sync();
        // stage 3: the k-th largest key among the C candidates (NS slots of 64)
        auto resolve = [&](auto ns_tag) {
          constexpr int NS = decltype(ns_tag)::value;
          uint32_t ck[NS], ci[NS];
          float cf[NS];
          bool ok[NS];
#pragma unroll
          for (int r = 0; r < NS; ++r) {
            const uint32_t j = lane + kWave * r;
            ok[r] = j < C;
            cf[r] = ok[r] ? cval[j] : 0.0f;
            ci[r] = ok[r] ? cidx[j] : 0u;
            ck[r] = ok[r] ? key_of(cf[r]) : 0u;
          }
          // The search stops early once exactly k candidates are >= the
          // threshold so far: those are then the k largest.  Below L the
          // candidate count is not the block's, hence c >= L.  (The
          // remaining steps are skipped by a uniform test rather than left
          // by a loop exit, which keeps the control flow simple.)
          uint32_t t = 0;
          bool exact = false;
#pragma unroll
          for (int bit = 30; bit >= 0; --bit) {
            if (!exact) {
              const uint32_t c = t | (1u << bit);
              uint32_t n = 0;
#pragma unroll
              for (int r = 0; r < NS; ++r) n += popc(ballot(ck[r] >= c));
              if (n >= (uint32_t)kq) {
                t = c;
                exact = n == (uint32_t)kq && c >= Lb;
              }
            }
          }
          T = t;
          uint32_t ngt = 0, neq = 0;
          if (!exact) {
#pragma unroll
            for (int r = 0; r < NS; ++r) {
              ngt += popc(ballot(ok[r] && ck[r] > t));
              neq += popc(ballot(ok[r] && ck[r] == t));
            }
          }
          // exact: every key >= t is kept; else the keys above t and the
          // first `need` keys equal to t in element order
          const uint32_t need = exact ? 0u : (uint32_t)kq - ngt;
          notie = exact || neq == need;
          uint32_t eq_before = 0, sel_before = 0;
#pragma unroll
          for (int r = 0; r < NS; ++r) {
            const bool gt = ok[r] && (exact ? ck[r] >= t : ck[r] > t);
            const bool eq = !exact && ok[r] && ck[r] == t;
            const uint64_t em = ballot(eq);
            const uint32_t rank = eq_before + lanes_below(em);
            eq_before += popc(em);
            const uint64_t lm = ballot(eq && rank == need - 1);
            if (lm) i_last = __builtin_amdgcn_readlane(ci[r], (int)__builtin_ctzll(lm));
            const bool sel = gt || (eq && rank < need);
            const uint64_t sm = ballot(sel);
            if (sel) {
              const uint32_t w = ((row_lo - span_lo) >> 2) + (sel_before + lanes_below(sm)) * (EB / 4);
              const typename E::T x = E::make(ci[r], cf[r]);
              if constexpr (VF32) *(u32x2*)(rowbuf + w) = x;
              else rowbuf[w] = x;
            }
            sel_before += popc(sm);
          }
        };
        const uint32_t nslot = (C + kWave - 1) / kWave;
        if (nslot == 1) resolve(std::integral_constant<int, 1>{});
        else if (nslot == 2) resolve(std::integral_constant<int, 2>{});
        else resolve(std::integral_constant<int, 4>{});
        // the lines of the new row: the row from the resolve, the rest of
        // the first and last line as read
        if (edge_off < row_lo || edge_off >= row_hi) rowbuf[(edge_off - span_lo) >> 2] = edge_old;
        wave_sync();
        const uint32_t nvec4 = (span_hi - span_lo) >> 4;
        for (uint32_t q = (uint32_t)lane; q < nvec4; q += kWave)
          __builtin_amdgcn_raw_buffer_store_b128(*(const u32x4*)(rowbuf + 4 * q), rrec, span_lo + 16 * q, 0, 0);
      }
    }
  }
  if (general) {
    // Exact bitwise search over every element (ties, large k, many
    // candidates): the largest T with #{key >= T} >= k.  Keys are compared
    // as |a| against the float with the same bits (the same order for
    // finite values; the thresholds tried never exceed +inf's bits).
    uint32_t t = 0;
    bool exact = false;
    for (int bit = 30; bit >= 0 && !exact; --bit) {
      const uint32_t c = t | (1u << bit);
      const float cf = __uint_as_float(c);
      uint32_t n = 0;
#pragma unroll
      for (int v = 0; v < NV; ++v) {
#pragma unroll
        for (int e = 0; e < 8; ++e) n += popc(ballot(__builtin_fabsf(a[v][e]) >= cf));
        __builtin_amdgcn_sched_barrier(0);  // bounds the masks in flight
      }
      if (n >= (uint32_t)kq) {
        t = c;
        exact = n == (uint32_t)kq;
      }
    }
    T = t;
    // kept: with an exact count |a| >= t; else |a| > t, and |a| == t for the
    // first `need` such elements in element order
    uint32_t sel_l = 0;
    if (exact) {
      notie = true;
      const float tf = opaque_f(__uint_as_float(t));
#pragma unroll
      for (int v = 0; v < NV; ++v)
#pragma unroll
        for (int e = 0; e < 8; ++e) sel_l += __builtin_fabsf(a[v][e]) >= tf ? 1u : 0u;
    } else {
      const float tf = opaque_f(__uint_as_float(t));
      uint32_t ngt_l = 0, neq_l = 0;
#pragma unroll
      for (int v = 0; v < NV; ++v)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          ngt_l += __builtin_fabsf(a[v][e]) > tf ? 1u : 0u;
          neq_l += __builtin_fabsf(a[v][e]) == tf ? 1u : 0u;
        }
      uint32_t ngt = 0;
#pragma unroll
      for (int b2 = 0; b2 < 7; ++b2) ngt += popc(ballot((ngt_l >> b2) & 1u)) << b2;
      const uint32_t need = (uint32_t)kq - ngt;  // >= 1
      // keys equal to t in the lanes before this one
      uint32_t eq_pre = 0;
#pragma unroll
      for (int b2 = 0; b2 < 7; ++b2) eq_pre += lanes_below(ballot((neq_l >> b2) & 1u)) << b2;
      // the lane holding the need-th key equal to t finds its index
      const bool mine = eq_pre < need && eq_pre + neq_l >= need;
      uint32_t my_last = 0;
      if (mine) {
        const float tf2 = opaque_f(tf);
        uint32_t r = eq_pre;
#pragma unroll
        for (int v = 0; v < NV; ++v)
#pragma unroll
          for (int e = 0; e < 8; ++e)
            if (__builtin_fabsf(a[v][e]) == tf2) {
              if (r == need - 1) my_last = eb + 8 * v + e;
              ++r;
            }
      }
      const uint64_t mm = ballot(mine);
      i_last = __builtin_amdgcn_readlane(my_last, (int)__builtin_ctzll(mm));
      const int last_here = (int)i_last - (int)eb;
      const float tf3 = opaque_f(tf);
#pragma unroll
      for (int v = 0; v < NV; ++v)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float ab = __builtin_fabsf(a[v][e]);
          sel_l += ((ab > tf3) | ((ab == tf3) & (8 * v + e <= last_here))) ? 1u : 0u;
        }
    }
    // the kept elements of this lane, stored in element order
    uint32_t pos = 0;
#pragma unroll
    for (int b2 = 0; b2 < 7; ++b2) pos += lanes_below(ballot((sel_l >> b2) & 1u)) << b2;
    if (sel_l) {
      const float tf = opaque_f(__uint_as_float(t));
      const int last_here = notie ? (int)kWave * EPL : (int)i_last - (int)eb;
#pragma unroll
      for (int v = 0; v < NV; ++v)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float ab = __builtin_fabsf(a[v][e]);
          if ((ab > tf) | ((ab == tf) & (8 * v + e <= last_here))) {
            E::store(rw, row0 + pos, E::make(eb + 8 * v + e, a[v][e]));
            ++pos;
          }
        }
    }
  }

  // ---------------------------------------------- 4. e = Q(a with a[I] = 0)
  if constexpr (LQ) {
    lane_zero_kept<EPL>(a, T, notie, i_last, eb);
    lane_partials<EPL>(a, p, b, eb, rem, gb);
  } else {
    lane_quantize_store<EPL, LB, EFM>(a, T, notie, i_last, eb, s, rem, full, bl, wide, re, rs,
                                      EfStream{b.e0, b.j, (uint32_t)p.t, p.seed_lo, p.seed_hi});
  }
}

// One thread per bucket of the step (all tensors): the (min, max) over the
// partials of the blocks it covers, -0 stored as +0, into table t mod 2.
__global__ void __launch_bounds__(256) bucket_reduce_kernel(StepParams p) {
  const int64_t cg = (int64_t)block_id() * 256 + thread_id();
  if (cg >= p.total_buckets) return;
  const __attribute__((address_space(4))) TensorDesc* td = constant_ptr(p.tensors);
  int lo = 0, hi = p.n_tensors - 1;  // the last tensor whose buckets start at or before cg
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (td[mid].first_bucket <= cg) lo = mid;
    else hi = mid - 1;
  }
  const TensorDesc d = load_desc(td + lo);
  const int64_t bq = p.big_bucket, B = p.block;
  const int64_t c = cg - d.first_bucket;
  const int64_t e_lo = c * bq;
  const int64_t e_hi = e_lo + bq < d.numel ? e_lo + bq : d.numel;
  const int64_t q_lo = e_lo / B, q_hi = (e_hi - 1) / B;
  const Rsrc rp = make_rsrc(p.state + p.partial_plane, (uint32_t)(p.total_blocks * 16));
  float mn = __builtin_inff(), mx = -__builtin_inff();
  for (int64_t q = q_lo; q <= q_hi; ++q) {
    const int64_t gb = q == d.num_blocks - 1 ? d.last_block : d.first_block + q;
    const uint32_t part = (q * B) / bq == c ? 0u : 8u;  // the block's first bucket, or its second
    const u32x2 pr = __builtin_amdgcn_raw_buffer_load_b64(rp, (uint32_t)(gb * 16) + part, 0, 0);
    mn = __builtin_fminf(mn, __uint_as_float(pr[0]));
    mx = __builtin_fmaxf(mx, __uint_as_float(pr[1]));
  }
  mn = mn + 0.0f;  // a bucket bound of -0 is stored as +0
  mx = mx + 0.0f;
  const uint64_t t = (uint64_t)(p.t & 1);
  float* out = (float*)(p.state + p.stats_plane + t * p.table_bytes) + 2 * cg;
  out[0] = mn;
  out[1] = mx;
}

// e = Q(a with a[I] = 0) for buckets spanning blocks (Algorithm 1; Algorithm
// 2, Q; Lemma 1 with kEfRandom): recomputes a = g + Q^-1(e) exactly as the
// select kernel did (same codes, same pairs), zeroes the elements of the
// block's new window row, and quantizes with the new pairs.  One wave per
// block, 64 elements per lane.
template <bool GBF16, bool VF32, int EFM>
__global__ void __launch_bounds__(kWave) __attribute__((amdgpu_waves_per_eu(4)))
requant_kernel(StepParams p, int64_t first) {
  constexpr int EPL = 64, NV = EPL / 8, CAP = kWave * EPL;
  constexpr int CW = (EFM & kEf8) ? 2 : 1;
  using E = Entry<VF32>;
  __shared__ uint32_t kept[CAP / 32];  // bit i: element i is in the new row

  const int lane = thread_id();
  const uint32_t eb = (uint32_t)lane * EPL;
  const int64_t gb = first + block_id();
  const uint32_t ef_bytes = (EFM & kEf8) ? (uint32_t)p.block : (uint32_t)(p.block >> 1);
  const Rsrc re = make_rsrc(p.state + p.ef_plane + (uint64_t)gb * ef_bytes, ef_bytes);
  const bool wide = p.block == CAP;
  LaneIn<EPL, true, GBF16, EFM> in;
  lane_load_codes(in, re, eb, wide);
  const Block b = locate(p, gb);
  const int s = b.s, kq = b.kq;
  const bool full = s == CAP;
  const Rsrc rg = make_rsrc((const uint8_t*)b.desc.grad + b.e0 * (GBF16 ? 2 : 4), vec_bytes<GBF16>(s));
  lane_load_grad(in, rg, eb);
  const LqBuckets old_b = lq_buckets(p, b, eb, EPL, 0), new_b = lq_buckets(p, b, eb, EPL, 1);

  kept[lane] = 0u;
  kept[lane + kWave] = 0u;
  wave_sync();
  const Rsrc rw = window_rsrc<VF32 ? 2 : 1>(p, gb, kq);
  const uint32_t row0 = (uint32_t)p.new_slot * kq;
  for (int j = lane; j < kq; j += kWave) {
    const uint32_t i = E::idx(E::load(rw, row0 + j));
    atomicOr(&kept[(i >> 5) & (CAP / 32 - 1)], 1u << (i & 31));
  }
  wave_sync();

  float a[NV][8];
  const int rem = s - (int)eb;
  lane_decode_lq(in, old_b, a, rem, full);
  const uint32_t k0 = kept[2 * lane], k1 = kept[2 * lane + 1];  // this lane's 64 elements
#pragma unroll
  for (int v = 0; v < NV; ++v)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int i = 8 * v + e;
      const uint32_t bit = i < 32 ? (k0 >> i) & 1u : (k1 >> (i - 32)) & 1u;
      if (bit) a[v][e] = 0.0f;
    }

  const float lo0 = __uint_as_float(new_b.st[0][0]), u0 = ef_step<EFM>(__uint_as_float(new_b.st[0][1]) - lo0);
  const float lo1 = __uint_as_float(new_b.st[1][0]), u1 = ef_step<EFM>(__uint_as_float(new_b.st[1][1]) - lo1);
  const EfStream st{b.e0, b.j, (uint32_t)p.t, p.seed_lo, p.seed_hi};
  constexpr float L = (EFM & kEf8) ? 255.0f : 15.0f;
  uint32_t wv[NV * CW];
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    // each element against its own bucket's pair, with an IEEE division
    uint32_t w24[8] = {};
    if constexpr ((EFM & kEfRandom) != 0) philox_w24((uint64_t)(b.e0 + eb + 8 * v) >> 2, st, w24);
    uint32_t w[CW];
#pragma unroll
    for (int c = 0; c < CW; ++c) w[c] = 0;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const bool second = 8 * v + e >= new_b.sp;
      const float lo = second ? lo1 : lo0, u = second ? u1 : u0;
      uint32_t code = 0;
      if (u != 0.0f)
        code = (EFM & kEfRandom) ? code_randomized(a[v][e], lo, u, L, w24[e]) : code_nearest(a[v][e], lo, u, L);
      if (8 * v + e >= rem) code = 0;  // past the block's end
      if constexpr (EFM & kEf8) w[e >> 2] |= code << (8 * (e & 3));
      else w[0] |= code << (4 * e);
    }
#pragma unroll
    for (int c = 0; c < CW; ++c) wv[CW * v + c] = w[c];
  }
  if ((int)eb < s) lane_store_codes<EPL, EFM>(wv, eb, wide, re);
}

// ================================================ select, blocks above 4096
// NW waves per block (B_d <= NW*4096); thread t owns the 64 consecutive
// elements [64t, 64t + 64), so wave w holds the block's 4096-element
// sub-block w.  The k-th largest |a| comes from an exact bitwise search over
// the keys (|a| as integers) of a bracket [lo, hi) that holds it: fewer than
// k keys lie at or above hi, at least k at or above lo, and the at most
// 8 keys per thread between them are gathered in LDS, so every bit costs a
// few comparisons per thread and one barrier; once at most 256 keys remain
// undecided they are gathered again and the waves finish 4 bits per barrier
// (a 16-ary search, one digit per wave).  The bracket is read off a sample of
// 1024 keys (16-ary in the same way) and checked by one counting pass; when
// the check fails (an unlucky sample, large tie groups) a bitwise search over
// every element narrows it instead.  The new row is written in element order,
// and for each sub-block the position in the row of its first entry goes to
// the record's segment table, behind the m rows, where the update finds the
// entries of one sub-block.
constexpr int kSubBlock = 4096;
constexpr int kCandPerThread = 8;
template <bool B>
struct BoolTag {
  static constexpr bool value = B;
};
constexpr int kSamples = 1024;
constexpr int kSampleRes = 19;  // the sample's order statistics are taken to 2^19 (1/16 of a binade)

template <int NW>
struct LargeLds {
  // counts [2][NW], scan totals [2][NW], bracket counts [2][NW], misc [4],
  // digit counts [2][2][16], the last keys [256], and the sample (kSamples)
  // or the gathered keys (NC + a sink word per lane)
  static constexpr size_t region() {
    return (size_t)NW * kWave * kCandPerThread + kWave > (size_t)kSamples ? (size_t)NW * kWave * kCandPerThread + kWave
                                                                          : (size_t)kSamples;
  }
  static constexpr size_t words() { return (size_t)6 * NW + 4 + 64 + 256 + region(); }
};

template <int NW, bool LB, bool GBF16, bool VF32>
__global__ void __launch_bounds__(NW * kWave) select_large_kernel(StepParams p, int64_t first) {
  constexpr int EPL = 64, NV = 8, NT = NW * kWave, CAP = NT * EPL, R = kCandPerThread, NC = NT * R;
  constexpr int SPT = kSamples / NT, SPL = kSamples / kWave;  // samples per thread; per lane
  constexpr int DPW = 16 / NW;                                  // sample digits per wave
  static_assert(SPT >= 1 && SPT <= NV, "one to eight samples per thread");
  using E = Entry<VF32>;
  extern __shared__ __align__(16) uint32_t smem[];
  uint32_t* const cnt = smem;           // [2][NW] per-wave counts, alternating between searches
  uint32_t* const pre = cnt + 2 * NW;   // [2][NW] per-wave totals of the two element-order scans
  uint32_t* const two = pre + 2 * NW;   // [2][NW] per-wave counts of a bracket pass
  uint32_t* const misc = two + 2 * NW;  // [4]
  uint32_t* const dig = misc + 4;       // [2][32] counts per digit, alternating between rounds
  uint32_t* const last = dig + 64;      // [256] the last undecided keys
  uint32_t* const region = last + 256;  // the sample, then the gathered keys

  const int tid = thread_id(), lane = tid & (kWave - 1), wave = (int)sgpr((uint32_t)tid / kWave);
  const uint32_t eb = (uint32_t)tid * EPL;
  const int bl = p.bucket_log2;
  const int64_t gb = first + block_id();

  const uint32_t nbk = (uint32_t)(p.block >> bl);
  const Rsrc re = make_rsrc(p.state + p.ef_plane + (uint64_t)gb * (p.block >> 1), (uint32_t)(p.block >> 1));
  const Rsrc rs = make_rsrc(p.state + p.stats_plane + (uint64_t)gb * nbk * 8, nbk * 8);
  const bool wide = p.block == CAP;
  LaneIn<EPL, LB, GBF16> in;
  lane_load_state(in, re, rs, eb, bl, wide);
  const Block b = locate(p, gb);
  const int s = b.s, kq = b.kq;
  const bool full = s == CAP;
  const Rsrc rg = make_rsrc((const uint8_t*)b.desc.grad + b.e0 * (GBF16 ? 2 : 4), vec_bytes<GBF16>(s));
  lane_load_grad(in, rg, eb);

  // ---------------------------------------------- 1. a = g + Q^-1(e)
  float a[NV][8];
  const int rem = s - (int)eb;
  lane_decode(in, a, rem, full);

  // workgroup sum of one value per wave; `buf` alternates between calls
  auto wg_sum = [&](uint32_t wave_value, int buf) {
    if (lane == 0) cnt[buf * NW + wave] = wave_value;
    lds_sync();
    uint32_t t = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) t += cnt[buf * NW + w];
    return sgpr(t);
  };
  // exclusive prefix in element order of a per-thread count below 128, and
  // the workgroup total; `slot` selects one of the two scan buffers
  auto wg_scan = [&](uint32_t c, int slot, uint32_t& total) {
    uint32_t in_wave = 0, wave_total = 0;
#pragma unroll
    for (int b2 = 0; b2 < 7; ++b2) {
      const uint64_t m = ballot((c >> b2) & 1u);
      in_wave += lanes_below(m) << b2;
      wave_total += popc(m) << b2;
    }
    if (lane == 0) pre[slot * NW + wave] = wave_total;
    lds_sync();
    uint32_t before = 0, all = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const uint32_t x = pre[slot * NW + w];
      all += x;
      before += w < wave ? x : 0u;
    }
    total = sgpr(all);
    return sgpr(before) + in_wave;
  };

  // ---------------------------------------------- 2. Top-K (exact search)
  // The bracket tests compare |a| as floats, which agrees with the keys as
  // integers except that a NaN reaches no bound (as in the comparisons of
  // (b)); an upper bound above the infinity pattern (2^31: none) is no bound,
  // and a lower bound there is never used.  Masks of whole waves: in
  // [lo1, hi) is (|a| >= lo1) and not (|a| >= hi).
  // (each caller passes bounds made opaque in its own branch, so that the
  // comparisons are not hoisted above it and kept for all elements at once)
  auto masks = [&](auto nohi_tag, float ab, float lof, float hif, uint64_t& m_in, uint64_t& m_hi) {
    const uint64_t ml = ballot(ab >= lof);
    if constexpr (decltype(nohi_tag)::value) {
      m_hi = 0;
      m_in = ml;
    } else {
      m_hi = ballot(ab >= hif);
      m_in = ml & ~m_hi;
    }
  };
  // keys in [lo1, hi) counted per thread (and their element-order positions
  // returned), keys >= hi counted for the workgroup; one barrier
  auto bracket_pass = [&](uint32_t lo1, uint32_t hi, uint32_t& n_hi, uint32_t& nc) {
    const float lof = __uint_as_float(lo1), hif = __uint_as_float(hi < 0x7F800000u ? hi : 0x7F800000u);
    uint32_t nh = 0, nc_l = 0;
    auto count = [&](auto nohi_tag) {
      const float lob = opaque_f(lof), hib = opaque_f(hif);
#pragma unroll
      for (int v = 0; v < NV; ++v) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          uint64_t m_in, m_hi;
          masks(nohi_tag, __builtin_fabsf(a[v][e]), lob, hib, m_in, m_hi);
          nh += popc(m_hi);
          nc_l += __builtin_amdgcn_inverse_ballot_w64(m_in) ? 1u : 0u;
        }
        nh = (uint32_t)opaque((int)nh);
      }
    };
    if (hi > 0x7F800000u)
      count(BoolTag<true>{});
    else
      count(BoolTag<false>{});
    uint32_t in_wave = 0, wave_total = 0;
#pragma unroll
    for (int b2 = 0; b2 < 7; ++b2) {
      const uint64_t m = ballot((nc_l >> b2) & 1u);
      in_wave += lanes_below(m) << b2;
      wave_total += popc(m) << b2;
    }
    if (lane == 0) {
      two[wave] = nh;
      two[NW + wave] = wave_total;
    }
    lds_sync();
    uint32_t all_h = 0, all_c = 0, before = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      all_h += two[w];
      const uint32_t x = two[NW + w];
      all_c += x;
      before += w < wave ? x : 0u;
    }
    n_hi = sgpr(all_h);
    nc = sgpr(all_c);
    return sgpr(before) + in_wave;
  };

  uint32_t lo = 0, hi = 1u << 31, n_hi = 0, nc = 0, pos = 0;
  bool narrowed = false;  // [lo, hi) holds the answer and at most NC keys; pos, nc, n_hi hold
  if (s > NC) {
    // (a) a bracket from the sample: one key per 8-element group, at the
    // group's element lane mod 8; the ranks around the expected rank
    // ns * kq / s of the answer, three standard deviations apart
#pragma unroll
    for (int i = 0; i < SPT; ++i) {
      float x = a[i][0];
#pragma unroll
      for (int e = 1; e < 8; ++e) x = (lane & 7) == e ? a[i][e] : x;
      region[tid * SPT + i] = 8 * i + (lane & 7) < rem ? __float_as_uint(x) & 0x7FFFFFFFu : 0u;
    }
    lds_sync();
    // samples that lie in the block: SPT per thread below s / 64, and those
    // of the thread holding the block's end
    const int r = s & 63, o = (s >> 6) & 7;
    const int part = r > o ? (r - o + 7) >> 3 : 0;
    const int ns = SPT * (s >> 6) + (part < SPT ? part : SPT);
    // (approximate arithmetic: the bracket is checked exactly below)
    const float mu = (float)ns * (float)kq * __builtin_amdgcn_rcpf((float)s);
    const float sd = 3.0f * __builtin_amdgcn_sqrtf(mu);
    const int r_lo = (int)__builtin_ceilf(mu + sd), r_hi = (int)__builtin_floorf(mu - sd);
    uint32_t key[SPL];
#pragma unroll
    for (int j = 0; j < SPL; ++j) key[j] = region[lane + kWave * j];
    // the largest 12-bit prefixes tl, th (bits 30..19) with at least r_lo,
    // r_hi samples at or above them; wave w counts digits w*DPW + i >= 1
    uint32_t tl = 0, th = 0;
#pragma unroll
    for (int rd = 0; rd < 3; ++rd) {
      const int sh = 27 - 4 * rd;
      uint32_t* const dg = dig + (rd & 1) * 32;
#pragma unroll
      for (int i = 0; i < DPW; ++i) {
        const uint32_t d = (uint32_t)(wave * DPW + i);
        if (d == 0) continue;
        const uint32_t cl = tl + (d << sh), ch = th + (d << sh);
        uint32_t nl = 0, nh = 0;
#pragma unroll
        for (int j = 0; j < SPL; ++j) {
          nl += popc(ballot(key[j] >= cl));
          nh += popc(ballot(key[j] >= ch));
        }
        if (lane == 0) {
          dg[d] = nl;
          dg[16 + d] = nh;
        }
      }
      lds_sync();
      const uint32_t x = lane < 32 ? dg[lane] : 0u;
      const uint32_t dl = popc(ballot(lane >= 1 && lane < 16 && x >= (uint32_t)r_lo));
      const uint32_t dh = popc(ballot(lane >= 17 && lane < 32 && (int)x >= r_hi));
      tl += dl << sh;
      th += dh << sh;
    }
    lo = r_lo > ns ? 0u : tl;
    hi = r_hi < 1 ? 1u << 31 : th + (1u << kSampleRes);
    if (lo <= 0x7F800000u) {  // else the sample was mostly NaN
      pos = bracket_pass(lo > 1u ? lo : 1u, hi, n_hi, nc);
      narrowed = n_hi < (uint32_t)kq && n_hi + nc >= (uint32_t)kq && nc <= (uint32_t)NC;
    }
  }

  uint32_t t = 0;
  bool exact = false;
  int buf = 0;
  if (!narrowed) {
    // (b) bitwise search over every element.  Before bit b the answer lies in
    // [t, U) with U = t + 2^(b+1); n_t keys (at most) are >= t, n_hi keys are
    // >= U, fewer than kq.  It stops once [t, U) holds at most NC keys.
    uint32_t U = 1u << 31, n_t = (uint32_t)s;
    n_hi = 0;
    int bit = 30;
    for (; bit >= 0 && !exact && n_t - n_hi > (uint32_t)NC; --bit) {
      const uint32_t c = t | (1u << bit);
      const float cf = __uint_as_float(c);
      uint32_t n = 0;
#pragma unroll
      for (int v = 0; v < NV; ++v) {
#pragma unroll
        for (int e = 0; e < 8; ++e) n += popc(ballot(__builtin_fabsf(a[v][e]) >= cf));
        n = (uint32_t)opaque((int)n);  // counted here: at most 8 masks in flight
      }
      n = wg_sum(n, buf);
      buf ^= 1;
      if (n >= (uint32_t)kq) {
        t = c;
        n_t = n;
        exact = n == (uint32_t)kq;
      } else {
        U = c;
        n_hi = n;
      }
    }
    if (bit >= 0 && !exact) {
      lo = t;
      hi = U;
      pos = bracket_pass(t > 1u ? t : 1u, U, n_hi, nc);  // nc <= n_t - n_hi <= NC
      narrowed = true;
    }
  }
  if (narrowed) {
    // (c) gather the keys in [max(lo, 1), hi) (0 never counts), then search
    // them bit by bit: a prefix c >= hi fails and a prefix c <= lo passes
    // without counting; otherwise count(|a| >= c) = n_hi + the gathered
    // keys >= c
    const uint32_t lo1 = lo > 1u ? lo : 1u;
    {
      // (pos stays below nc <= NC; the others write a sink word per lane)
      const float lof = __uint_as_float(lo1), hif = __uint_as_float(hi < 0x7F800000u ? hi : 0x7F800000u);
      auto gather = [&](auto nohi_tag) {
        const float lob = opaque_f(lof), hib = opaque_f(hif);
#pragma unroll
        for (int v = 0; v < NV; ++v) {
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            uint64_t m_in, m_hi;
            masks(nohi_tag, __builtin_fabsf(a[v][e]), lob, hib, m_in, m_hi);
            const bool inb = __builtin_amdgcn_inverse_ballot_w64(m_in);
            region[inb ? pos : (uint32_t)(NC + lane)] = __float_as_uint(a[v][e]);
            pos += inb ? 1u : 0u;
          }
          __builtin_amdgcn_sched_barrier(0);  // one vector's stores at a time
        }
      };
      if (hi > 0x7F800000u)
        gather(BoolTag<true>{});
      else
        gather(BoolTag<false>{});
    }
    lds_sync();
    uint32_t y[R];  // the keys: |a| as integers
#pragma unroll
    for (int r = 0; r < R; ++r) y[r] = (uint32_t)(tid + r * NT) < nc ? region[tid + r * NT] & 0x7FFFFFFFu : 0u;
    // [max(t, lo1), U) holds n_t - n_u undecided keys: n_t = count(>= max(t, lo1)),
    // n_u = count(>= U); a prefix c >= U fails without counting
    t = 0;
    uint32_t U = hi, n_t = n_hi + nc, n_u = n_hi;
    int bit = 30;
    for (; bit >= 0 && !exact && n_t - n_u > 256u; --bit) {
      const uint32_t c = t | (1u << bit);
      if (c >= U) continue;
      if (c <= lo) {
        t = c;
        continue;
      }
      uint32_t n = 0;
#pragma unroll
      for (int r = 0; r < R; ++r) n += popc(ballot(y[r] >= c));
      n = n_hi + wg_sum((uint32_t)opaque((int)n), buf);  // n_hi: the keys >= hi
      buf ^= 1;
      if (n >= (uint32_t)kq) {
        t = c;
        n_t = n;
        exact = n == (uint32_t)kq;
      } else {
        U = c;
        n_u = n;
      }
    }
    if (bit >= 0 && !exact) {
      // the at most 256 undecided keys go to `last`; the remaining bits are
      // found 4 at a time: wave w counts count(>= t + (d << sh)) for its
      // digits d = w*DPW + i >= 1 as n_u + the keys in `last` >= that prefix
      const uint32_t t1 = t > lo1 ? t : lo1;
      uint32_t m_l = 0;
#pragma unroll
      for (int r = 0; r < R; ++r) m_l += (y[r] >= t1) & (y[r] < U) ? 1u : 0u;
      uint32_t nl;
      uint32_t q = wg_scan(m_l, 0, nl);
#pragma unroll
      for (int r = 0; r < R; ++r)
        if ((y[r] >= t1) & (y[r] < U)) last[q++ & 255u] = y[r];
      lds_sync();
      uint32_t z[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) z[i] = (uint32_t)(lane + kWave * i) < nl ? last[lane + kWave * i] : 0u;
      for (int rd = 0; bit >= 0 && !exact; ++rd) {
        const int width = bit >= 3 ? 4 : bit + 1;
        const int sh = bit + 1 - width;
        const uint32_t nd = 1u << width;  // digits 0 .. nd - 1
        uint32_t* const dg = dig + (rd & 1) * 32;
#pragma unroll
        for (int i = 0; i < DPW; ++i) {
          const uint32_t d = (uint32_t)(wave * DPW + i);
          if (d == 0) continue;
          const uint32_t c = t + (d << sh);
          uint32_t n;
          if (d >= nd || c >= U) {
            n = 0u;  // fails
          } else if (c <= lo) {
            n = ~0u;  // passes, count not needed
          } else {
            n = n_u;
#pragma unroll
            for (int j = 0; j < 4; ++j) n += popc(ballot(z[j] >= c));
          }
          if (lane == 0) dg[d] = n;
        }
        lds_sync();
        const uint32_t x = lane < 16 ? dg[lane] : 0u;
        const uint64_t pass = ballot(lane >= 1 && lane < 16 && x >= (uint32_t)kq);
        const uint32_t dstar = popc(pass);  // counts fall with the digit
        const uint32_t n_at = sgpr(__builtin_amdgcn_readlane(x, (int)dstar));
        if (dstar + 1 < nd) {
          const uint32_t cu = t + ((dstar + 1) << sh);
          U = cu < U ? cu : U;
        }
        t += dstar << sh;
        exact = dstar >= 1 && n_at == (uint32_t)kq;
        bit = sh - 1;
      }
    }
  }
  const uint32_t T = t;
  uint32_t i_last = 0;
  bool notie = exact;
  uint32_t sel_l = 0;
  if (exact) {
    const float tf = opaque_f(__uint_as_float(t));
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
      for (int e = 0; e < 8; ++e) sel_l += __builtin_fabsf(a[v][e]) >= tf ? 1u : 0u;
  } else {
    // the keys above t are kept, then the first `need` keys equal to t in
    // element order
    const float tf = opaque_f(__uint_as_float(t));
    uint32_t ngt_l = 0, neq_l = 0;
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        ngt_l += __builtin_fabsf(a[v][e]) > tf ? 1u : 0u;
        neq_l += __builtin_fabsf(a[v][e]) == tf ? 1u : 0u;
      }
    uint32_t ngt_w = 0;
#pragma unroll
    for (int b2 = 0; b2 < 7; ++b2) ngt_w += popc(ballot((ngt_l >> b2) & 1u)) << b2;
    const uint32_t need = (uint32_t)kq - wg_sum(ngt_w, buf);  // >= 1
    uint32_t neq_all;
    const uint32_t eq_pre = wg_scan(neq_l, 0, neq_all);
    if (eq_pre < need && eq_pre + neq_l >= need) {  // the thread holding the need-th equal key
      const float tf2 = opaque_f(tf);
      uint32_t r = eq_pre, my_last = 0;
#pragma unroll
      for (int v = 0; v < NV; ++v)
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if (__builtin_fabsf(a[v][e]) == tf2) {
            if (r == need - 1) my_last = eb + 8 * v + e;
            ++r;
          }
      misc[0] = my_last;
    }
    lds_sync();
    i_last = sgpr(misc[0]);
    notie = neq_all == need;
    const int last_here = (int)i_last - (int)eb;
    const float tf3 = opaque_f(tf);
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float ab = __builtin_fabsf(a[v][e]);
        sel_l += ((ab > tf3) | ((ab == tf3) & (8 * v + e <= last_here))) ? 1u : 0u;
      }
  }
  {
    // the new row in element order, and the segment table entry of this
    // wave's sub-block: the row position of its first entry
    uint32_t kept_all;
    uint32_t pos = wg_scan(sel_l, 1, kept_all);
    constexpr uint32_t EB = VF32 ? 8u : 4u;
    const int nsub = (p.block + kSubBlock - 1) / kSubBlock;
    const Rsrc rrec = make_rsrc(p.state + p.win_plane + (uint64_t)gb * p.win_stride, (uint32_t)p.win_stride);
    if (lane == 0 && wave < nsub)
      __builtin_amdgcn_raw_buffer_store_b32(pos, rrec,
                                            (uint32_t)p.window * p.k_full * EB + ((uint32_t)p.new_slot * nsub + wave) * 4,
                                            0, 0);
    if (sel_l) {
      const Rsrc rw = window_rsrc<VF32 ? 2 : 1>(p, gb, kq);
      const uint32_t row0 = (uint32_t)p.new_slot * kq;
      const float tf = opaque_f(__uint_as_float(T));
      const int last_here = notie ? CAP : (int)i_last - (int)eb;
#pragma unroll
      for (int v = 0; v < NV; ++v) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float ab = __builtin_fabsf(a[v][e]);
          if ((ab > tf) | ((ab == tf) & (8 * v + e <= last_here))) {
            E::store(rw, row0 + pos, E::make(eb + 8 * v + e, a[v][e]));
            ++pos;
          }
        }
        __builtin_amdgcn_sched_barrier(0);  // one vector's stores at a time
      }
    }
  }

  // ---------------------------------------------- 4. e = Q(a with a[I] = 0)
  lane_quantize_store<EPL, LB>(a, T, notie, i_last, eb, s, rem, full, bl, wide, re, rs);
}

// ================================================ update, blocks above 4096
// One workgroup of 256 threads per 4096-element sub-block j of a block
// (thread tid: the sub-block's elements 16*tid + [0, 16)).  The live rows'
// entries of sub-block j are the segments the select kernel recorded.  The
// workgroup rebuilds z1 = sum beta1^r V and z2 = sum beta2^r V^2 one row at a
// time, oldest first (Algorithm 2, AdamStats), from registers when every row
// holds at most 256 of the sub-block's entries (and at most kFastRows rows are
// live), else from LDS, where they are staged in batches of stage_large
// entries.  Every thread then turns its own 16 elements' sums into the update
// (an element without entries has sums 0 and a decrement of 0) and applies it
// (Algorithm 1; Algorithm 4).  The staging batch is small (1024 entries, 512
// with binary32 values: 37 KB of LDS in all), so that four workgroups fit a
// compute unit for the register path, which uses no staging.
template <bool VF>
constexpr int stage_large() { return VF ? 512 : 1024; }
// Live rows up to which the update reads a sub-block's entries straight into
// registers (when no row holds more than 256 of them).
constexpr int kFastRows = 24;

template <bool VF>
constexpr size_t update_large_lds_bytes() {
  return (size_t)2 * (kSubBlock + kWave) * 4 + (size_t)3 * kWave * 4 + 16 + (size_t)stage_large<VF>() * (VF ? 8 : 4);
}

template <bool PBF16, bool VF32, bool EXPORT>
__global__ void __launch_bounds__(256) update_large_kernel(StepParams p, int64_t first_block, int32_t nsub,
                                                           float* mhat, float* vhat) {
  constexpr int NT = 256, STAGE = stage_large<VF32>();
  using E = Entry<VF32>;
  using ET = typename E::T;
  extern __shared__ __align__(16) uint32_t smem[];
  float* const z1 = (float*)smem;                         // [kSubBlock] + sink words
  float* const z2 = z1 + kSubBlock + kWave;
  uint32_t* const seg_lo = (uint32_t*)(z2 + kSubBlock + kWave);  // [kWave] by row age
  uint32_t* const seg_n = seg_lo + kWave;
  uint32_t* const seg_at = seg_n + kWave;  // position of the row's first entry in the staged order
  uint32_t* const misc = seg_at + kWave;   // [4]: the entry total, the longest segment
  ET* const stage = (ET*)(misc + 4);       // [STAGE]

  const int tid = thread_id(), lane = tid & (kWave - 1), wave = (int)sgpr((uint32_t)tid / kWave);
  const int64_t wg = block_id();
  const int32_t gb = (int32_t)(first_block + wg / nsub);
  const int j = (int)(wg % nsub);
  const Span g = span_of(p, gb, PBF16 ? 2 : 4);
  const int lo = j * kSubBlock;
  if (lo >= g.s) return;  // a sub-block past the end of a ragged block
  const int s = g.s - lo < kSubBlock ? g.s - lo : kSubBlock;
  const int kq = g.kq, m = p.window, n_live = p.n_live;
  const int slot0 = (p.new_slot + 1 + m - n_live) % m;  // oldest live row first
  const int nsub_blk = (p.block + kSubBlock - 1) / kSubBlock;  // table entries per row
  const uint32_t eb = (uint32_t)tid * 16;

  // the parameters go out first; their latency hides behind the rebuild
  const int es = PBF16 ? 2 : 4;
  const Rsrc rp = make_rsrc((const void*)(g.base + (uint64_t)lo * es), vec_bytes<PBF16>(s));
  Raw8<PBF16> th[2];
  if (!EXPORT) {
#pragma unroll
    for (int v = 0; v < 2; ++v) th[v] = load8<PBF16>(rp, eb + 8 * v);
  }

  // the live rows' segments of sub-block j (row age r = 0 is the oldest),
  // their starts in the staged order by a scan over wave 0's lanes
  constexpr uint32_t EB = VF32 ? 8u : 4u;
  const Rsrc rrec = make_rsrc(p.state + p.win_plane + (uint64_t)gb * p.win_stride, (uint32_t)p.win_stride);
  const uint32_t table = (uint32_t)m * p.k_full * EB;
  if (wave == 0) {
    uint32_t n = 0, start = 0;
    if (lane < n_live) {
      const int slot = (slot0 + lane) % m;
      const uint32_t a0 = __builtin_amdgcn_raw_buffer_load_b32(rrec, table + ((uint32_t)slot * nsub_blk + j) * 4, 0, 0);
      const uint32_t a1 = j + 1 < nsub_blk
                              ? __builtin_amdgcn_raw_buffer_load_b32(rrec, table + ((uint32_t)slot * nsub_blk + j + 1) * 4, 0, 0)
                              : (uint32_t)kq;
      start = (uint32_t)slot * kq + a0;  // entry number in the record
      n = a1 - a0;
    }
    uint32_t inc = n, big = n;  // inclusive prefix over lanes; the longest segment
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
      const uint32_t o = __shfl_up(inc, d, kWave);
      if (lane >= d) inc += o;
      const uint32_t b2 = __shfl_xor(big, d, kWave);
      big = b2 > big ? b2 : big;
    }
    seg_lo[lane] = start;
    seg_n[lane] = n;
    seg_at[lane] = inc - n;
    if (lane == kWave - 1) {
      misc[0] = inc;
      misc[1] = big;
    }
  }
  {
    const float4 zero = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      *(float4*)(z1 + eb + 4 * q) = zero;
      *(float4*)(z2 + eb + 4 * q) = zero;
    }
  }
  lds_sync();
  const uint32_t total = misc[0];

  const Rsrc rw = window_rsrc<VF32 ? 2 : 1>(p, gb, kq);
  const float w1s = lane < kMaxWindow ? constant_ptr(p.wpow)[lane] : 0.0f;
  const float w2s = lane < kMaxWindow ? constant_ptr(p.wpow)[kMaxWindow + lane] : 0.0f;
  // one workgroup-wide read-add-write of a row's entry per thread (the
  // entries of a row have distinct indices)
  auto add_entry = [&](ET e, float w1, float w2) {
    const uint32_t i = E::idx(e) - (uint32_t)lo;
    const uint32_t zp = i < (uint32_t)s ? i : (uint32_t)(kSubBlock + lane);
    const float v = E::val(e);
    const float a1 = z1[zp], a2 = z2[zp];
    z1[zp] = a1 + w1 * v;
    z2[zp] = a2 + w2 * (v * v);
  };
  if (n_live <= kFastRows && misc[1] <= (uint32_t)NT) {
    // every live row holds at most NT entries of the sub-block: thread t
    // loads entry t of every row at once, then the rows are added oldest
    // first from registers, a barrier between rows
    ET ld[kFastRows];
#pragma unroll
    for (int r = 0; r < kFastRows; ++r)
      if (r < n_live && (uint32_t)tid < seg_n[r]) ld[r] = E::load(rw, seg_lo[r] + (uint32_t)tid);
#pragma unroll
    for (int r = 0; r < kFastRows; ++r) {
      const uint32_t n = r < n_live ? seg_n[r] : 0u;
      if (n != 0) {  // (uniform)
        const int age = n_live - 1 - r;
        const float w1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(w1s), age));
        const float w2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(w2s), age));
        if ((uint32_t)tid < n) add_entry(ld[r], w1, w2);
        lds_sync();
      }
    }
  } else
  for (uint32_t b0 = 0; b0 < total; b0 += STAGE) {
    const uint32_t b1 = total - b0 < (uint32_t)STAGE ? total : b0 + STAGE;
    // stage the entries [b0, b1) of the concatenated segments: every thread
    // issues the loads of its positions b0 + tid + NT*i together (the row of
    // a position by binary search over the rows' first positions), then
    // writes them to LDS
    {
      constexpr int PER = STAGE / NT;
      ET ld[PER];
#pragma unroll
      for (int i = 0; i < PER; ++i) {
        const uint32_t x = b0 + tid + NT * i;
        int r = 0;
        for (int half = 32; half > 0; half >>= 1)
          if (r + half < n_live && seg_at[r + half] <= x) r += half;
        const uint32_t entry = x < b1 ? seg_lo[r] + (x - seg_at[r]) : 0u;
        ld[i] = E::load(rw, entry);
      }
#pragma unroll
      for (int i = 0; i < PER; ++i)
        if (b0 + tid + NT * i < b1) stage[tid + NT * i] = ld[i];
    }
    lds_sync();
    // row by row, oldest first, the whole workgroup on one row: a row's
    // entries have distinct indices, so its read-add-writes never meet; a
    // barrier orders them before the next row's (the summation order per
    // element is the rows' order, as with one wave)
    for (int r = 0; r < n_live; ++r) {
      const uint32_t at = seg_at[r], n = seg_n[r];
      const uint32_t x0 = at > b0 ? at : b0, x1 = at + n < b1 ? at + n : b1;
      const int age = n_live - 1 - r;
      const float w1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(w1s), age));
      const float w2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(w2s), age));
      for (uint32_t x = x0 + (uint32_t)tid; x < x1; x += NT) add_entry(stage[x - b0], w1, w2);
      lds_sync();
    }
  }
  float s1[16], s2[16];
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const float4 u1 = *(const float4*)(z1 + eb + 4 * q);
    const float4 u2 = *(const float4*)(z2 + eb + 4 * q);
    s1[4 * q] = u1.x; s1[4 * q + 1] = u1.y; s1[4 * q + 2] = u1.z; s1[4 * q + 3] = u1.w;
    s2[4 * q] = u2.x; s2[4 * q + 1] = u2.y; s2[4 * q + 2] = u2.z; s2[4 * q + 3] = u2.w;
  }

  // every thread: its 16 elements
  if ((int)eb >= s) return;
  if (EXPORT) {
#pragma unroll
    for (int e = 0; e < 16; ++e)
      if ((int)eb + e < s) {
        mhat[g.e0 + lo + eb + e] = p.c1 * s1[e];
        vhat[g.e0 + lo + eb + e] = p.c2 * s2[e];
      }
    return;
  }
  const bool full = s == kSubBlock;
#pragma unroll
  for (int v = 0; v < 2; ++v) {
    float thf[8], out[8];
    unpack8<PBF16>(th[v], thf);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float mh = p.c1 * s1[8 * v + e];
      const float vh = p.c2 * s2[8 * v + e];
      const float den = p.eps + __builtin_amdgcn_sqrtf(vh);
      // an element without entries is left to the decay alone
      const bool none = (s1[8 * v + e] == 0.0f) & (s2[8 * v + e] == 0.0f);
      const float d = none ? 0.0f : p.lr * (mh * __builtin_amdgcn_rcpf(den));
      const float base = p.decay_is_one ? thf[e] : thf[e] * p.decay;
      out[e] = base - d;
    }
    store8<PBF16>(rp, eb + 8 * v, s, full, out);
  }
}

// ============================================================ update
// The accumulators hold, per element of the block, sum beta1^r V and sum
// beta2^r V^2 (z1 and z2; or z1 alone, one after the other), then z1 the
// parameter decrement.  Element i lives at word
// ((i >> 2) & 3) * 4*NT + (i >> 4) * 4 + (i & 3), so that the 16 elements of a
// thread are four 16-byte words at a stride of 4*NT words and a wave's
// 16-byte accesses fall on consecutive addresses.  Word CAP of each array is
// a sink for lanes without an entry, which keeps the sparse updates free of
// branches.
template <int NT>
__device__ __forceinline__ uint32_t zpos(uint32_t i) {
  return ((i >> 2) & 3u) * (4u * NT) + (i >> 4) * 4u + (i & 3u);
}

// Staged window positions of the update kernel: KC chunks of 64, rounded up
// to whole multiples of the workgroup so that every thread stages the same
// count.
template <int NT, int KC>
constexpr int update_stage_entries() { return (KC * kWave + NT - 1) / NT * NT; }

// LDS: the accumulators (two, or one with ONE), then the staged window
// entries in chunk order.
template <int NT, bool VF, int KC, bool ONE>
constexpr size_t update_lds_bytes() {
  return (size_t)(ONE ? 1 : 2) * (NT * kLaneElems + 16) * 4 + (size_t)update_stage_entries<NT, KC>() * (VF ? 8 : 4);
}

// One workgroup per block.  One wave (rotating with the block) rebuilds the
// moments of the block's window entries, oldest row first, and turns them
// into parameter decrements; then every thread updates its own elements.
//
// Window entries are staged in LDS in the order the leader wave reads them:
// position q = 64*c + lane of chunk c, where chunk c is part c mod R of the
// live row c / R (oldest row first, R = ceil(k_q/64) parts of 64 entries),
// each with its index replaced by its accumulator word (the sink word CAP for
// positions without an entry).  A block whose live rows need more than KC
// chunks is read by the leader straight from the window record.
//
// ONE = true: one accumulator; the leader makes two passes over the staged
// entries (first moments, read back and cleared, then second moments), which
// halves the LDS of a workgroup so that eight fit on a compute unit.  The
// host launches it only where every block's live rows fit in KC chunks.
// ONE = false: two accumulators, any block.  EXPORT = true writes dense m-hat
// and v-hat instead of updating theta.
// Waves per SIMD that the LDS of an update workgroup allows (160 KB per
// compute unit, four SIMDs); telling the compiler lets it spend registers
// up to that occupancy on keeping LDS reads in flight.
template <int NT, bool VF, int KC, bool ONE>
constexpr int update_waves_per_eu() {
  const int per_cu = (int)(163840 / update_lds_bytes<NT, VF, KC, ONE>());
  const int w = per_cu * (NT / kWave) / 4;
  return w < 1 ? 1 : w > 8 ? 8 : w;
}

template <int NT, bool PBF16, bool VF32, bool EXPORT, int KC, bool ONE>
__global__ void __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(update_waves_per_eu<NT, VF32, KC, ONE>())))
update_kernel(StepParams p, int64_t first_block, float* mhat, float* vhat) {
  static_assert(!ONE || !EXPORT, "one accumulator: parameter update only");
  constexpr int NW = NT / kWave;
  constexpr int CAP = NT * kLaneElems;
  constexpr int kChunks = KC;                             // 64-entry chunks the leader holds
  constexpr int NP = update_stage_entries<NT, KC>() / NT;  // staged positions per thread
  using E = Entry<VF32>;
  using ET = typename E::T;
  extern __shared__ __align__(16) uint32_t smem[];
  float* const z1 = (float*)smem;
  float* const z2 = z1 + CAP + 16;                        // not allocated with ONE
  ET* const stage = (ET*)(ONE ? z2 : z2 + CAP + 16);      // [NP * NT]; chunks past KC are not read

  const int tid = thread_id(), lane = tid & (kWave - 1), wave = (int)sgpr(tid / kWave);
  const uint32_t eb = (uint32_t)tid * kLaneElems;
  const int m = p.window, n_live = p.n_live;
  // oldest live row first: the row written at step s is slot (s-1) mod m
  const int slot0 = (p.new_slot + 1 + m - n_live) % m;

  const Span u = span_of(p, (int32_t)(first_block + block_id()), PBF16 ? 2 : 4);
  const int s = u.s, kq = u.kq;
  const int leader = u.gb & (NW - 1);
  const int R = (kq + kWave - 1) / kWave;
  const float rcp_r = 1.0f / (float)R;
  const bool staged = n_live * R <= kChunks;

  // chunk c -> (live row, part): the entry of staged position q, and whether
  // it holds one (uniform per block: kq, R, n_live)
  auto position = [&](int q, uint32_t& entry) {
    const int c = q >> 6;
    const int row = (int)(((float)c + 0.5f) * rcp_r);  // c / R for c < 2^10
    const int jj = (c - row * R) * kWave + (q & (kWave - 1));
    int slot = slot0 + row;
    if (slot >= m) slot -= m;
    const bool valid = row < n_live && jj < kq;
    entry = valid ? (uint32_t)(slot * kq + jj) : 0u;
    return valid;
  };

  // loads: window positions (unconditional; positions without an entry read
  // entry 0 and are not used), then the parameters
  const Rsrc rw = window_rsrc<VF32 ? 2 : 1>(p, u.gb, kq);
  ET w[NP];
#pragma unroll
  for (int i = 0; i < NP; ++i) {
    uint32_t entry;
    position(tid + NT * i, entry);
    w[i] = E::load(rw, entry);
  }
  const Rsrc rp = make_rsrc((const void*)u.base, vec_bytes<PBF16>(s));
  Raw8<PBF16> th[2];
  if (!EXPORT) {
#pragma unroll
    for (int v = 0; v < 2; ++v) th[v] = load8<PBF16>(rp, eb + v * 8);
  }
  const float w1s = lane < kMaxWindow ? constant_ptr(p.wpow)[lane] : 0.0f;
  const float w2s = lane < kMaxWindow ? constant_ptr(p.wpow)[kMaxWindow + lane] : 0.0f;

  {
    const float4 zero = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      *(float4*)(z1 + q * 4 * NT + tid * 4) = zero;
      if (!ONE) *(float4*)(z2 + q * 4 * NT + tid * 4) = zero;
    }
  }
#pragma unroll
  for (int i = 0; i < NP; ++i) {
    const int q = tid + NT * i;
    uint32_t entry;
    const bool valid = position(q, entry);
    const uint32_t idx = E::idx(w[i]);
    const uint32_t zw = valid && idx < (uint32_t)s ? zpos<NT>(idx) : (uint32_t)CAP;
    stage[q] = E::with_word(w[i], zw);
  }
  lds_sync();

  if (wave == leader) {
    auto step_of = [&](float s1, float s2) {
      const float mh = p.c1 * s1;
      const float vh = p.c2 * s2;
      const float den = p.eps + __builtin_amdgcn_sqrtf(vh);
      return p.lr * (mh * __builtin_amdgcn_rcpf(den));
    };
    if (staged) {
      // chunks past the live rows hold only sink words
      uint32_t zp[kChunks];
      float val[kChunks];
      int rr[kChunks];
      {
        int row = 0, col = 0;
#pragma unroll
        for (int c = 0; c < kChunks; ++c) {
          const ET x = stage[c * kWave + lane];
          zp[c] = E::word(x);
          val[c] = E::val(x);
          rr[c] = (n_live - 1 - row) & (kMaxWindow - 1);
          if (++col == R) {
            col = 0;
            ++row;
          }
        }
      }
      // The entries of one row (or of one 64-entry part of it) have distinct
      // indices, so each chunk reads, adds and writes back its words (the
      // sink word's lanes race harmlessly); chunks follow each other oldest
      // row first.  Every entry's sums are read before any word is
      // overwritten, so an index that occurs in several rows gets the same
      // decrement from each occurrence.
      if constexpr (ONE) {
#pragma unroll
        for (int c = 0; c < kChunks; ++c) {
          const float w1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(w1s), rr[c]));
          const float a1 = z1[zp[c]];
          z1[zp[c]] = a1 + w1 * val[c];
        }
        float s1[kChunks];
#pragma unroll
        for (int c = 0; c < kChunks; ++c) s1[c] = z1[zp[c]];
#pragma unroll
        for (int c = 0; c < kChunks; ++c) z1[zp[c]] = 0.0f;
#pragma unroll
        for (int c = 0; c < kChunks; ++c) {
          const float w2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(w2s), rr[c]));
          const float vv = val[c] * val[c];
          const float a2 = z1[zp[c]];
          z1[zp[c]] = a2 + w2 * vv;
        }
        float d[kChunks];
#pragma unroll
        for (int c = 0; c < kChunks; ++c) d[c] = step_of(s1[c], z1[zp[c]]);
#pragma unroll
        for (int c = 0; c < kChunks; ++c) z1[zp[c]] = d[c];
      } else {
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
          float d[kChunks];
#pragma unroll
          for (int c = 0; c < kChunks; ++c) d[c] = step_of(z1[zp[c]], z2[zp[c]]);
#pragma unroll
          for (int c = 0; c < kChunks; ++c) z1[zp[c]] = d[c];
        }
      }
    } else if constexpr (!ONE) {
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
          mhat[u.e0 + i] = p.c1 * a1[r];
          vhat[u.e0 + i] = p.c2 * a2[r];
        }
      }
    }
    return;
  }

  // ------------------------------------------------ 6. parameter update
  const bool full = s == NT * kLaneElems;
#pragma unroll
  for (int v = 0; v < 2; ++v) {
    const uint32_t e0 = eb + v * 8;   // vectors past s store nothing
    const float4 u0 = *(const float4*)(z1 + (2 * v) * 4 * NT + tid * 4);
    const float4 u1 = *(const float4*)(z1 + (2 * v + 1) * 4 * NT + tid * 4);
    const float upd[8] = {u0.x, u0.y, u0.z, u0.w, u1.x, u1.y, u1.z, u1.w};
    float thf[8], out[8];
    unpack8<PBF16>(th[v], thf);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float base = p.decay_is_one ? thf[e] : thf[e] * p.decay;
      out[e] = base - upd[e];
    }
    store8<PBF16>(rp, e0, s, full, out);
  }
}

template <int EPL, bool LB, bool GB, bool VF, int EFM>
hipError_t launch_select_t(const StepParams& p, int64_t first, int64_t count, hipStream_t stream) {
  if (count <= 0) return hipSuccess;
  const size_t lds = select_lds_words() * 4;
  hipLaunchKernelGGL((select_kernel<EPL, LB, GB, VF, EFM>), dim3((uint32_t)count), dim3(kWave), lds, stream, p,
                     first);
  return hipGetLastError();
}

// Elements per lane of the select kernel: 16, 32 or 64.
inline int select_epl(int block) { return block <= 1024 ? 16 : block <= 2048 ? 32 : 64; }

// Waves of the large-block select kernel: 4096 elements each, 2 to 16.
inline int large_waves(int block) {
  const int w = (block + kSubBlock - 1) / kSubBlock;
  return w <= 2 ? 2 : w <= 4 ? 4 : w <= 8 ? 8 : 16;
}

template <int NW, bool GB, bool VF>
hipError_t launch_select_large_t(const StepParams& p, int64_t first, int64_t count, hipStream_t stream) {
  if (count <= 0) return hipSuccess;
  const size_t lds = LargeLds<NW>::words() * 4;
  if ((1 << p.bucket_log2) >= 64)
    hipLaunchKernelGGL((select_large_kernel<NW, true, GB, VF>), dim3((uint32_t)count), dim3(NW * kWave), lds, stream,
                       p, first);
  else
    hipLaunchKernelGGL((select_large_kernel<NW, false, GB, VF>), dim3((uint32_t)count), dim3(NW * kWave), lds,
                       stream, p, first);
  return hipGetLastError();
}

template <bool GB, bool VF>
hipError_t launch_select_large(const StepParams& p, int64_t first, int64_t count, hipStream_t stream) {
  switch (large_waves(p.block)) {
    case 2: return launch_select_large_t<2, GB, VF>(p, first, count, stream);
    case 4: return launch_select_large_t<4, GB, VF>(p, first, count, stream);
    case 8: return launch_select_large_t<8, GB, VF>(p, first, count, stream);
    default: return launch_select_large_t<16, GB, VF>(p, first, count, stream);
  }
}

// One workgroup per 4096-element sub-block of each block of [first, first + count).
template <bool PB, bool VF, bool EXPORT>
hipError_t launch_update_large(const StepParams& p, int64_t first, int64_t count, float* mh, float* vh,
                               hipStream_t stream) {
  if (count <= 0) return hipSuccess;
  const int32_t nsub = (p.block + kSubBlock - 1) / kSubBlock;
  hipLaunchKernelGGL((update_large_kernel<PB, VF, EXPORT>), dim3((uint32_t)(count * nsub)), dim3(256),
                     update_large_lds_bytes<VF>(), stream, p, first, nsub, mh, vh);
  return hipGetLastError();
}

template <int EPL, bool GB, bool VF, int EFM>
hipError_t launch_select_e(const StepParams& p, int64_t first, int64_t count, hipStream_t stream) {
  // whole buckets per lane (B_q >= EPL) or buckets of whole vectors
  if ((1 << p.bucket_log2) >= EPL) return launch_select_t<EPL, true, GB, VF, EFM>(p, first, count, stream);
  return launch_select_t<EPL, false, GB, VF, EFM>(p, first, count, stream);
}

// Blocks above 4096 elements take the multi-wave kernel, which has the
// default code format only (the host rejects the others there).
template <bool GB, bool VF, int EFM>
hipError_t launch_select_d(const StepParams& p, int64_t first, int64_t count, hipStream_t stream) {
  if (p.block > kSubBlock) {
    if constexpr (EFM != 0) return hipErrorInvalidValue;
    else return launch_select_large<GB, VF>(p, first, count, stream);
  }
  switch (select_epl(p.block)) {
    case 16: return launch_select_e<16, GB, VF, EFM>(p, first, count, stream);
    case 32: return launch_select_e<32, GB, VF, EFM>(p, first, count, stream);
    default: return launch_select_e<64, GB, VF, EFM>(p, first, count, stream);
  }
}

template <bool GB, bool VF>
hipError_t launch_select_f(const StepParams& p, int64_t first, int64_t count, hipStream_t stream) {
  switch (p.ef_mode) {
    case 0: return launch_select_d<GB, VF, 0>(p, first, count, stream);
    case kEf8: return launch_select_d<GB, VF, kEf8>(p, first, count, stream);
    case kEfRandom: return launch_select_d<GB, VF, kEfRandom>(p, first, count, stream);
    case kEf8 | kEfRandom: return launch_select_d<GB, VF, kEf8 | kEfRandom>(p, first, count, stream);
    default: return hipErrorInvalidValue;
  }
}

// Chunks of 64 window entries the update's leader wave processes per block:
// the live rows of a full block rounded up to 4, 8, 10, 12 or 16.
inline int chunk_class(const StepParams& p) {
  const int R = (p.k_full + kWave - 1) / kWave;
  const int nch = p.n_live * R;
  return nch <= 4 ? 4 : nch <= 8 ? 8 : nch <= 10 ? 10 : nch <= 12 ? 12 : 16;
}

template <int NT, bool PB, bool VF, int KC, bool ONE>
hipError_t launch_update_k(const StepParams& p, int64_t first, int64_t count, hipStream_t stream) {
  if (count <= 0) return hipSuccess;
  const size_t lds = update_lds_bytes<NT, VF, KC, ONE>();
  hipLaunchKernelGGL((update_kernel<NT, PB, VF, false, KC, ONE>), dim3((uint32_t)count), dim3(NT), lds, stream, p,
                     first, (float*)nullptr, (float*)nullptr);
  return hipGetLastError();
}

// Blocks [first, first + count), one workgroup each: with one accumulator
// where the live rows of a full block, and so of every block, fit in 16
// chunks; else with two.
template <int NT, bool PB, bool VF>
hipError_t launch_update_t(const StepParams& p, int64_t first, int64_t count, hipStream_t stream) {
  const int R = (p.k_full + kWave - 1) / kWave;
  if (p.n_live * R > 16) return launch_update_k<NT, PB, VF, 16, false>(p, first, count, stream);
  switch (chunk_class(p)) {
    case 4: return launch_update_k<NT, PB, VF, 4, true>(p, first, count, stream);
    case 8: return launch_update_k<NT, PB, VF, 8, true>(p, first, count, stream);
    case 10: return launch_update_k<NT, PB, VF, 10, true>(p, first, count, stream);
    case 12: return launch_update_k<NT, PB, VF, 12, true>(p, first, count, stream);
    default: return launch_update_k<NT, PB, VF, 16, true>(p, first, count, stream);
  }
}

template <int NT, bool VF>
hipError_t launch_export(const StepParams& p, int64_t first_block, int64_t blocks, float* mh, float* vh,
                         hipStream_t stream) {
  if (blocks <= 0) return hipSuccess;
  const size_t lds = update_lds_bytes<NT, VF, 16, false>();
  hipLaunchKernelGGL((update_kernel<NT, false, VF, true, 16, false>), dim3((uint32_t)blocks), dim3(NT), lds, stream,
                     p, first_block, mh, vh);
  return hipGetLastError();
}

template <bool GB, bool VF, int EF8>
hipError_t launch_select_partials_t(const StepParams& p, hipStream_t stream) {
  const size_t lds = select_lds_words() * 4;
  hipLaunchKernelGGL((select_kernel<64, true, GB, VF, EF8, true>), dim3((uint32_t)p.total_blocks), dim3(kWave), lds,
                     stream, p, (int64_t)0);
  return hipGetLastError();
}

template <bool GB, bool VF>
hipError_t launch_select_partials_d(const StepParams& p, hipStream_t stream) {
  return (p.ef_mode & kEf8) ? launch_select_partials_t<GB, VF, kEf8>(p, stream)
                            : launch_select_partials_t<GB, VF, 0>(p, stream);
}

template <bool GB, bool VF, int EFM>
hipError_t launch_requant_t(const StepParams& p, hipStream_t stream) {
  hipLaunchKernelGGL((requant_kernel<GB, VF, EFM>), dim3((uint32_t)p.total_blocks), dim3(kWave), 0, stream, p,
                     (int64_t)0);
  return hipGetLastError();
}

template <bool GB, bool VF>
hipError_t launch_requant_d(const StepParams& p, hipStream_t stream) {
  switch (p.ef_mode) {
    case 0: return launch_requant_t<GB, VF, 0>(p, stream);
    case kEf8: return launch_requant_t<GB, VF, kEf8>(p, stream);
    case kEfRandom: return launch_requant_t<GB, VF, kEfRandom>(p, stream);
    case kEf8 | kEfRandom: return launch_requant_t<GB, VF, kEf8 | kEfRandom>(p, stream);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

size_t step_lds_bytes(int block, int k_full, int value_f32) {
  (void)k_full;
  (void)value_f32;
  const int nt = threads_for_block(block);
  if (block > kSubBlock) return update_large_lds_bytes<true>();
  const size_t sel = select_lds_words() * 4;
  const size_t upd = nt == 64 ? update_lds_bytes<64, true, 16, false>() : update_lds_bytes<256, true, 16, false>();
  return sel > upd ? sel : upd;
}

hipError_t launch_select(const StepParams& p, int grad_bf16, int value_f32, int64_t first, int64_t count,
                         hipStream_t stream) {
  if (grad_bf16)
    return value_f32 ? launch_select_f<true, true>(p, first, count, stream)
                     : launch_select_f<true, false>(p, first, count, stream);
  return value_f32 ? launch_select_f<false, true>(p, first, count, stream)
                   : launch_select_f<false, false>(p, first, count, stream);
}

hipError_t launch_update(const StepParams& p, int param_bf16, int value_f32, int64_t first, int64_t count,
                         hipStream_t stream) {
  if (p.block > kSubBlock) {
    if (param_bf16)
      return value_f32 ? launch_update_large<true, true, false>(p, first, count, nullptr, nullptr, stream)
                       : launch_update_large<true, false, false>(p, first, count, nullptr, nullptr, stream);
    return value_f32 ? launch_update_large<false, true, false>(p, first, count, nullptr, nullptr, stream)
                     : launch_update_large<false, false, false>(p, first, count, nullptr, nullptr, stream);
  }
  if (threads_for_block(p.block) == 64) {
    if (param_bf16)
      return value_f32 ? launch_update_t<64, true, true>(p, first, count, stream)
                       : launch_update_t<64, true, false>(p, first, count, stream);
    return value_f32 ? launch_update_t<64, false, true>(p, first, count, stream)
                     : launch_update_t<64, false, false>(p, first, count, stream);
  }
  if (param_bf16)
    return value_f32 ? launch_update_t<256, true, true>(p, first, count, stream)
                     : launch_update_t<256, true, false>(p, first, count, stream);
  return value_f32 ? launch_update_t<256, false, true>(p, first, count, stream)
                   : launch_update_t<256, false, false>(p, first, count, stream);
}

hipError_t launch_moments(const StepParams& p, int64_t first_block, int64_t num_blocks, float* mhat,
                          float* vhat, int value_f32, hipStream_t stream) {
  if (p.block > kSubBlock)
    return value_f32 ? launch_update_large<false, true, true>(p, first_block, num_blocks, mhat, vhat, stream)
                     : launch_update_large<false, false, true>(p, first_block, num_blocks, mhat, vhat, stream);
  if (threads_for_block(p.block) == 64)
    return value_f32 ? launch_export<64, true>(p, first_block, num_blocks, mhat, vhat, stream)
                     : launch_export<64, false>(p, first_block, num_blocks, mhat, vhat, stream);
  return value_f32 ? launch_export<256, true>(p, first_block, num_blocks, mhat, vhat, stream)
                   : launch_export<256, false>(p, first_block, num_blocks, mhat, vhat, stream);
}

hipError_t launch_select_partials(const StepParams& p, int grad_bf16, int value_f32, hipStream_t stream) {
  if (p.total_blocks <= 0) return hipSuccess;
  if (grad_bf16)
    return value_f32 ? launch_select_partials_d<true, true>(p, stream) : launch_select_partials_d<true, false>(p, stream);
  return value_f32 ? launch_select_partials_d<false, true>(p, stream) : launch_select_partials_d<false, false>(p, stream);
}

hipError_t launch_bucket_reduce(const StepParams& p, hipStream_t stream) {
  if (p.total_buckets <= 0) return hipSuccess;
  const uint32_t grid = (uint32_t)((p.total_buckets + 255) / 256);
  hipLaunchKernelGGL(bucket_reduce_kernel, dim3(grid), dim3(256), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_requant(const StepParams& p, int grad_bf16, int value_f32, hipStream_t stream) {
  if (p.total_blocks <= 0) return hipSuccess;
  if (grad_bf16)
    return value_f32 ? launch_requant_d<true, true>(p, stream) : launch_requant_d<true, false>(p, stream);
  return value_f32 ? launch_requant_d<false, true>(p, stream) : launch_requant_d<false, false>(p, stream);
}

}  // namespace microadam
