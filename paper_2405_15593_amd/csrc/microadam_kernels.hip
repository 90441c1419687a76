// MicroAdam step kernels for CDNA4 (gfx950).
//
// The step kernel is persistent: each workgroup owns a contiguous range of
// Top-K blocks (B_d elements of one tensor each) and, for each block, runs
// the whole step of Algorithm 1 in one pass over HBM while the inputs of its
// next block are already in flight:
//   1. a = g + Q^-1(e)                            (Algorithm 1; Algorithm 2, Q^-1)
//   2. block Top-K of |a|, lower index wins ties   (Section 3.1, "Top-K")
//   3. a[I] = 0; bucket (delta, Delta) = (min, max) by lane shuffles;
//      e = Q(a, delta, Delta), two 4-bit codes per byte  (Algorithm 1; Section 3.1)
//   4. the new window row (I, bf16(V)) is stored   (Section 3.2)
//   5. m-hat, v-hat rebuilt in LDS from the window rows with weights
//      beta^(t-s)                                  (Algorithm 2, AdamStats)
//   6. theta <- (1 - eta*lambda) theta - eta m / (eps + sqrt(v))
//                                                  (Algorithm 1; Algorithm 4)
// Blocks share nothing, so workgroups never communicate.
//
// Element layout inside a block: thread `tid` of NT owns two vectors of 8
// consecutive elements; vector v holds elements v*NT*8 + tid*8 + [0, 8).  Each
// wave-wide load or store instruction covers one contiguous span, and an EF
// bucket of B_q elements is held by B_q/8 neighbouring lanes.
//
// Arithmetic that decides an integer (EF decode, accumulator, Top-K order,
// bucket min/max, codes) is binary32 with one rounding per written operation
// (the file is compiled with -ffp-contract=off); the only fused operations in
// that part are in div15, which is exact, and the code brackets of step 3,
// which are checked against the exact quotient's rounding.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

#include "microadam_device.h"

namespace microadam {
namespace {

constexpr int kWave = 64;
constexpr int NV = 2;                // vectors of 8 elements per thread
constexpr int kRegion = 32;          // candidate vectors one wave can hand to wave 0
constexpr int kCand = 256;           // candidate elements wave 0 resolves
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

template <int CTRL>
__device__ __forceinline__ float dpp_mov(float x) {
  return __builtin_bit_cast(
      float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xF, 0xF, false));
}

// min / max over groups of G neighbouring lanes (G a power of two <= 64).
__device__ __forceinline__ void group_minmax(float& mn, float& mx, int G) {
  if (G > 1) { mn = __builtin_fminf(mn, dpp_mov<0xB1>(mn)); mx = __builtin_fmaxf(mx, dpp_mov<0xB1>(mx)); }
  if (G > 2) { mn = __builtin_fminf(mn, dpp_mov<0x4E>(mn)); mx = __builtin_fmaxf(mx, dpp_mov<0x4E>(mx)); }
  if (G > 4) { mn = __builtin_fminf(mn, dpp_mov<0x141>(mn)); mx = __builtin_fmaxf(mx, dpp_mov<0x141>(mx)); }
  if (G > 8) { mn = __builtin_fminf(mn, dpp_mov<0x140>(mn)); mx = __builtin_fmaxf(mx, dpp_mov<0x140>(mx)); }
  for (int off = 16; off < G; off <<= 1) {
    mn = __builtin_fminf(mn, __shfl_xor(mn, off, kWave));
    mx = __builtin_fmaxf(mx, __shfl_xor(mx, off, kWave));
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
  r.ef_off = d->ef_off;
  r.stats_off = d->stats_off;
  r.win_off = d->win_off;
  r.k_full = d->k_full;
  r.k_last = d->k_last;
  return r;
}

__device__ __forceinline__ uint32_t key_of(float a) { return __float_as_uint(a) & 0x7FFFFFFFu; }

// Workgroup barrier that orders LDS only.  The waves of a workgroup exchange
// data through LDS alone, so no wait for outstanding global loads or stores
// (in particular the next block's prefetch) is needed here.
__device__ __forceinline__ void lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// -------------------------------------------------------- element vectors
// Raw storage of 8 consecutive elements of a bf16 or float32 tensor.
template <bool BF16> struct Raw8 { u32x4 w[BF16 ? 1 : 2]; };

// Vector loads only: the resource covers the block rounded up to whole
// 8-element vectors.  A 16-byte-aligned vector that holds a valid element
// never crosses the end of a page-aligned mapping, so the few elements read
// past the end of a ragged tensor are harmless; they are masked to 0 by the
// caller.
template <bool BF16>
__device__ __forceinline__ Raw8<BF16> load8(Rsrc r, uint32_t elem) {
  Raw8<BF16> x;
  constexpr uint32_t es = BF16 ? 2 : 4;
  x.w[0] = __builtin_amdgcn_raw_buffer_load_b128(r, elem * es, 0, 0);
  if constexpr (!BF16) x.w[1] = __builtin_amdgcn_raw_buffer_load_b128(r, elem * es + 16, 0, 0);
  return x;
}

// bytes covered by the vectors of a block of s elements
template <bool BF16>
__device__ __forceinline__ uint32_t vec_bytes(int s) {
  return (((uint32_t)s + 7u) & ~7u) * (BF16 ? 2u : 4u);
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
  static constexpr int kWords = VF32 ? 2 : 1;
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
  __device__ static T lds_get(const uint32_t* base, uint32_t entry) {
    if constexpr (VF32) return *(const u32x2*)(base + 2 * entry);
    else return base[entry];
  }
  __device__ static void lds_put(uint32_t* base, uint32_t entry, T e) {
    if constexpr (VF32) *(u32x2*)(base + 2 * entry) = e;
    else base[entry] = e;
  }
};

// ------------------------------------------------------- block geometry
struct Block {
  const uint8_t* grad;    // first element of the block
  uint8_t* param;
  uint8_t* ef;            // EF codes of the block
  uint8_t* stats;         // (delta, Delta) pairs of the block
  uint8_t* win;           // m window rows of the block
  int s;                  // valid elements
  int kq;                 // window entries per row
};

template <bool PBF16, bool GBF16, int EW>
__device__ __forceinline__ Block make_block(const StepParams& p, const TensorDesc& d, int64_t q) {
  Block b;
  const int64_t e0 = q * p.block;
  const int64_t rem = d.numel - e0;
  b.s = (int)(rem < p.block ? rem : p.block);
  b.kq = (q == d.num_blocks - 1) ? d.k_last : d.k_full;
  b.grad = (const uint8_t*)d.grad + e0 * (GBF16 ? 2 : 4);
  b.param = (uint8_t*)d.param + e0 * (PBF16 ? 2 : 4);
  b.ef = p.state + d.ef_off + (e0 >> 1);
  b.stats = p.state + d.stats_off + ((e0 >> p.bucket_log2) << 3);
  b.win = p.state + d.win_off + (uint64_t)q * p.window * d.k_full * EW * 4;
  return b;
}

// Inputs prefetched one block ahead.
template <bool GBF16> struct Prefetch {
  Raw8<GBF16> g[NV];
  uint32_t codes[NV];
  u32x2 st[NV];
};

template <int NT, bool GBF16>
__device__ __forceinline__ Prefetch<GBF16> prefetch(const Block& b, int bucket_log2) {
  Prefetch<GBF16> x;
  const int tid = threadIdx.x;
  const Rsrc rg = make_rsrc(b.grad, vec_bytes<GBF16>(b.s));
  const Rsrc re = make_rsrc(b.ef, (((uint32_t)b.s + 1) / 2 + 3) & ~3u);
  const uint32_t nbk = ((uint32_t)b.s + (1u << bucket_log2) - 1) >> bucket_log2;
  const Rsrc rs = make_rsrc(b.stats, nbk * 8);
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    const uint32_t i0 = v * NT * 8 + tid * 8;
    x.st[v] = __builtin_amdgcn_raw_buffer_load_b64(rs, (i0 >> bucket_log2) * 8, 0, 0);
    x.codes[v] = __builtin_amdgcn_raw_buffer_load_b32(re, i0 >> 1, 0, 0);
    x.g[v] = load8<GBF16>(rg, i0);
  }
  return x;
}

// ------------------------------------------------------- LDS carve-up
// Older window rows wave 0 holds in registers for the rebuild: up to this
// many chunks of 64 entries (a row of k entries takes ceil(k/64) chunks).
template <bool VF32> constexpr int stage_chunks() { return VF32 ? 4 : 9; }

template <int NT>
struct Lds {
  static constexpr int NW = NT / kWave;
  static constexpr int CAP = NT * 16;
  float* z1;          // [CAP] sum of beta1^r V, then the parameter decrement
  float* z2;          // [CAP] sum of beta2^r V^2, then -1 once converted
  float* regv;        // [NW][kRegion][8] candidate vectors per wave
  uint32_t* regi;     // [NW][kRegion] their first element index
  float* cval;        // candidate values (first half of regv, once read)
  uint32_t* cidx;     // candidate indices (second half of regv, once read)
  uint32_t* misc;     // 64 words: counts, wave bounds, broadcast, reductions
  uint32_t* newrow;   // [k_full entries] row written at step t
  __device__ Lds(uint32_t* smem) {
    z1 = (float*)smem;
    z2 = z1 + CAP;
    regv = z2 + CAP;
    regi = (uint32_t*)(regv + NW * kRegion * 8);
    cval = regv;
    cidx = (uint32_t*)(regv + NW * kRegion * 4);
    misc = regi + NW * kRegion;
    newrow = misc + 64;
  }
};
// misc word offsets
enum { M_COUNT = 0 /* [2*NW] */, M_WL = 8 /* [NW] */, M_GEN = 12, M_T = 13, M_ILAST = 14,
       M_NOTIE = 15, M_RED0 = 16, M_RED1 = 32, M_RED2 = 48 /* 16 words each */ };

template <int NT>
constexpr size_t lds_words(int k_full, int ew) {
  return 2 * (size_t)(NT * 16) + (size_t)(NT / kWave) * kRegion * 9 + 64 + (size_t)k_full * ew;
}

// Exclusive prefix, in element order, of per-(thread, vector) counts < 16.
// Returns the workgroup total; base[v] = counted elements before this thread's
// vector v.  One barrier; `red` (2*NW words) must not be reused until a later
// barrier.
template <int NT>
__device__ __forceinline__ uint32_t wg_scan(const uint32_t (&cnt)[NV], uint32_t (&base)[NV], uint32_t* red) {
  constexpr int NW = NT / kWave;
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  uint32_t pre[NV];
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    const uint64_t b0 = ballot(cnt[v] & 1u), b1 = ballot(cnt[v] & 2u);
    const uint64_t b2 = ballot(cnt[v] & 4u), b3 = ballot(cnt[v] & 8u);
    pre[v] = lanes_below(b0) + 2u * lanes_below(b1) + 4u * lanes_below(b2) + 8u * lanes_below(b3);
    if (lane == 0) red[v * NW + wave] = popc(b0) + 2u * popc(b1) + 4u * popc(b2) + 8u * popc(b3);
  }
  lds_sync();
  uint32_t run = 0;
#pragma unroll
  for (int v = 0; v < NV; ++v) {
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const uint32_t x = red[v * NW + w];
      if (w == wave) base[v] = run + pre[v];
      run += x;
    }
  }
  return run;
}

// Workgroup-wide count of elements flagged in NV 8-bit masks.  One barrier;
// consecutive calls must use different `red` buffers (NW words).
template <int NT>
__device__ __forceinline__ uint32_t wg_count(const uint32_t (&mask)[NV], uint32_t* red) {
  constexpr int NW = NT / kWave;
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
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

// ================================================================== step
template <int NT, bool PBF16, bool GBF16, bool VF32>
__device__ __forceinline__ void step_body(const StepParams& p) {
  constexpr int NW = NT / kWave;
  constexpr int CAP = NT * 16;
  constexpr int EW = VF32 ? 2 : 1;
  constexpr int kChunks = stage_chunks<VF32>();
  constexpr uint32_t kCandCap = (uint32_t)(kCand < NW * kRegion * 4 ? kCand : NW * kRegion * 4);
  using E = Entry<VF32>;
  using ET = typename E::T;
  extern __shared__ __align__(16) uint32_t smem[];
  const Lds<NT> l(smem);

  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const int bucket_log2 = p.bucket_log2;
  const int G = (1 << bucket_log2) >> 3;  // lanes per EF bucket

  // contiguous range of global blocks for this workgroup
  const int64_t NB = p.total_blocks, NG = gridDim.x, wg = blockIdx.x;
  const int64_t per = NB / NG, rem = NB % NG;
  int64_t gb = wg * per + (wg < rem ? wg : rem);
  const int64_t gb_end = gb + per + (wg < rem ? 1 : 0);
  if (gb >= gb_end) return;

  for (int x = tid * 4; x < 2 * CAP; x += NT * 4) *(float4*)(l.z1 + x) = make_float4(0.f, 0.f, 0.f, 0.f);

  // tensor cursor: the block whose inputs were prefetched last
  const auto* tensors = constant_ptr(p.tensors);
  uint32_t tj = constant_ptr(p.block_tensor)[gb];
  TensorDesc td = load_desc(tensors + tj);
  int64_t q = gb - td.first_block;
  Prefetch<GBF16> pre = prefetch<NT, GBF16>(make_block<PBF16, GBF16, EW>(p, td, q), bucket_log2);

  const int64_t t = p.t;
  const int n_old = p.n_old, m = p.window;
  // row slot of the oldest live row: (s - 1) mod m for s = t - n_old
  const int slot0 = (p.new_slot + m - n_old) % m;

  for (;;) {
    const Block cur = make_block<PBF16, GBF16, EW>(p, td, q);
    // ---------------------------------------------- next block's inputs
    // (the last block of the range prefetches itself again: no conditional
    // register copies)
    const bool has_next = gb + 1 < gb_end;
    if (has_next) {
      ++q;
      if (q == td.num_blocks) {
        ++tj;
        td = load_desc(tensors + tj);
        q = 0;
      }
    }
    const Prefetch<GBF16> npre = prefetch<NT, GBF16>(make_block<PBF16, GBF16, EW>(p, td, q), bucket_log2);

    const int s = cur.s, kq = cur.kq;
    const bool full = s == CAP;

    // ---------------------------------------------- 1. a = g + Q^-1(e)
    float a[NV][8];
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const float lo = __uint_as_float(pre.st[v][0]), hi = __uint_as_float(pre.st[v][1]);
      const float u = div15(hi - lo);
      const uint32_t w = pre.codes[v];
      const uint32_t ev = w & 0x0F0F0F0Fu, od = (w >> 4) & 0x0F0F0F0Fu;
      float g[8];
      unpack8<GBF16>(pre.g[v], g);
#pragma unroll
      for (int h = 0; h < 4; ++h) {  // v_cvt_f32_ubyte{0..3}
        const float c0 = (float)((ev >> (8 * h)) & 0xFFu);
        const float c1 = (float)((od >> (8 * h)) & 0xFFu);
        const float s0 = c0 * u, s1 = c1 * u;
        const float d0 = s0 + lo, d1 = s1 + lo;
        a[v][2 * h] = g[2 * h] + d0;
        a[v][2 * h + 1] = g[2 * h + 1] + d1;
      }
    }
    if (!full) {  // elements past the end of the tensor are 0 and never kept
#pragma unroll
      for (int v = 0; v < NV; ++v)
#pragma unroll
        for (int e = 0; e < 8; ++e)
          if ((int)(v * NT * 8 + tid * 8 + e) >= s) a[v][e] = 0.0f;
    }

    // ---------------------------------------------- 2. Top-K threshold
    // Lower bound L: per wave, the ceil(k/NW)-th largest lane maximum of |a|
    // (resolved on its top 13 bits); at least k elements are >= the minimum
    // over waves.
    float vmax[NV];
#pragma unroll
    for (int v = 0; v < NV; ++v) {
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

    // wave 0 fetches this block's older rows into registers (row i, oldest
    // first, in chunks i*R .. i*R+R-1 of 64 entries)
    const int R = (kq + kWave - 1) / kWave;
    const bool staged = n_old * R <= kChunks;
    const Rsrc rw = make_rsrc(cur.win, (uint32_t)(m * kq * EW * 4));
    ET stg[kChunks];
#pragma unroll
    for (int c = 0; c < kChunks; ++c) stg[c] = E::none();
    if (wave == 0 && staged) {
      int row = 0, col = 0, slot = slot0;
#pragma unroll
      for (int c = 0; c < kChunks; ++c) {
        if (row < n_old) {
          const int jj = col * kWave + lane;
          if (jj < kq) stg[c] = E::load(rw, slot * kq + jj);
        }
        if (++col == R) {
          col = 0;
          ++row;
          if (++slot == m) slot = 0;
        }
      }
    }

    float L;
    {
      uint32_t Lb = l.misc[M_WL];
#pragma unroll
      for (int w = 1; w < NW; ++w) Lb = min(Lb, l.misc[M_WL + w]);
      L = __uint_as_float(sgpr(Lb));
    }
    // candidate vectors: those holding some |a| >= L, handed to wave 0 in
    // element order (vector slot, wave, lane)
    {
      const uint64_t m0 = ballot(vmax[0] >= L), m1 = ballot(vmax[1] >= L);
      const uint32_t c0 = popc(m0);
      const uint32_t pos0 = lanes_below(m0), pos1 = c0 + lanes_below(m1);
      float* rv = l.regv + wave * kRegion * 8;
      uint32_t* ri = l.regi + wave * kRegion;
      if (vmax[0] >= L && pos0 < (uint32_t)kRegion) {
        *(float4*)(rv + pos0 * 8) = make_float4(a[0][0], a[0][1], a[0][2], a[0][3]);
        *(float4*)(rv + pos0 * 8 + 4) = make_float4(a[0][4], a[0][5], a[0][6], a[0][7]);
        ri[pos0] = tid * 8;
      }
      if (vmax[1] >= L && pos1 < (uint32_t)kRegion) {
        *(float4*)(rv + pos1 * 8) = make_float4(a[1][0], a[1][1], a[1][2], a[1][3]);
        *(float4*)(rv + pos1 * 8 + 4) = make_float4(a[1][4], a[1][5], a[1][6], a[1][7]);
        ri[pos1] = NT * 8 + tid * 8;
      }
      if (lane == 0) {
        l.misc[M_COUNT + wave] = c0;
        l.misc[M_COUNT + NW + wave] = popc(m1);
      }
    }
    lds_sync();  // B2 ------------------------------------------------

    // wave 0 resolves the threshold exactly among the candidates
    bool general;
    {
      uint32_t nvec = 0;
      bool overflow = false;
#pragma unroll
      for (int w = 0; w < NW; ++w) {
        const uint32_t c0 = sgpr(l.misc[M_COUNT + w]), c1 = sgpr(l.misc[M_COUNT + NW + w]);
        nvec += c0 + c1;
        overflow |= c0 + c1 > (uint32_t)kRegion;
      }
      general = !fast_k || L == 0.0f || overflow || nvec > 2u * kWave;
    }
    if (!general && wave == 0) {
      // this lane takes candidate vectors lane and lane + 64 (element order)
      uint32_t src[2];
      bool have[2];
#pragma unroll
      for (int r = 0; r < 2; ++r) {
        const uint32_t j = lane + kWave * r;
        uint32_t off = 0, at = 0;
        bool found = false;
#pragma unroll
        for (int i = 0; i < 2 * NW; ++i) {
          const int w = i % NW;
          const uint32_t ci = sgpr(l.misc[M_COUNT + i]);
          const uint32_t first = (i < NW) ? 0u : sgpr(l.misc[M_COUNT + w]);
          if (!found && j < off + ci) { found = true; at = w * kRegion + first + (j - off); }
          off += ci;
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
        for (int bit = 30; bit >= 0; --bit) {
          const uint32_t c = T | (1u << bit);
          uint32_t n = popc(ballot(ck[0] >= c));
          if (nslot > 1) n += popc(ballot(ck[1] >= c));
          if (nslot > 2) n += popc(ballot(ck[2] >= c));
          if (nslot > 3) n += popc(ballot(ck[3] >= c));
          if (n >= (uint32_t)kq) T = c;
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
          if (sel) {
            const ET ent = E::make(ci[r], cf[r]);
            E::store(rw, row0 + pos, ent);
            E::lds_put(l.newrow, pos, ent);
          }
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
        uint32_t mk[NV];
#pragma unroll
        for (int v = 0; v < NV; ++v) {
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
      uint32_t gtm[NV], eqm[NV];
#pragma unroll
      for (int v = 0; v < NV; ++v) {
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
      uint32_t ecnt[NV], ebase[NV];
#pragma unroll
      for (int v = 0; v < NV; ++v) ecnt[v] = __popc(eqm[v]);
      (void)wg_scan<NT>(ecnt, ebase, l.misc + (buf ? M_RED1 : M_RED0));
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        uint32_t r = ebase[v];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          if ((eqm[v] >> e) & 1u) {
            if (r == need - 1) l.misc[M_ILAST] = (uint32_t)(v * NT * 8 + tid * 8 + e);
            ++r;
          }
        }
      }
      lds_sync();
      i_last = sgpr(l.misc[M_ILAST]);
      notie = false;
      uint32_t scnt[NV], sbase[NV];
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        uint32_t c = 0;
#pragma unroll
        for (int e = 0; e < 8; ++e)
          c += ((gtm[v] >> e) & 1u) || (((eqm[v] >> e) & 1u) && (uint32_t)(v * NT * 8 + tid * 8 + e) <= i_last);
        scnt[v] = c;
      }
      (void)wg_scan<NT>(scnt, sbase, l.misc + M_RED2);
      const uint32_t row0 = (uint32_t)p.new_slot * kq;
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        uint32_t pos = sbase[v];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const uint32_t i = (uint32_t)(v * NT * 8 + tid * 8 + e);
          const bool sel = ((gtm[v] >> e) & 1u) || (((eqm[v] >> e) & 1u) && i <= i_last);
          if (sel) {
            const ET ent = E::make(i, a[v][e]);
            E::store(rw, row0 + pos, ent);
            E::lds_put(l.newrow, pos, ent);
            ++pos;
          }
        }
      }
      lds_sync();
    }

    // parameters of this block, needed after the quantization below
    const Rsrc rp = make_rsrc(cur.param, vec_bytes<PBF16>(s));
    Raw8<PBF16> th[NV];
#pragma unroll
    for (int v = 0; v < NV; ++v) th[v] = load8<PBF16>(rp, v * NT * 8 + tid * 8);

    // ---------------------------------------------- 5. moments (wave 0)
    // z1[idx] += beta1^r V and z2[idx] += beta2^r V^2 row by row, oldest
    // first; then every window index is converted once to the decrement
    // eta * m / (eps + sqrt(v)) (z2 = -1 marks a converted index).
    if (wave == 0) {
      const auto* w1 = constant_ptr(p.wpow);
      const auto* w2 = constant_ptr(p.wpow) + kMaxWindow;
      auto add = [&](ET e, int r) {
        const uint32_t idx = E::idx(e);
        if (idx < (uint32_t)s) {
          const float v = E::val(e);
          const float x1 = w1[r] * v;
          const float vv = v * v;
          const float x2 = w2[r] * vv;
          l.z1[idx] = l.z1[idx] + x1;
          l.z2[idx] = l.z2[idx] + x2;
        }
      };
      auto convert = [&](ET e) {
        const uint32_t idx = E::idx(e);
        if (idx < (uint32_t)s) {
          const float s2 = l.z2[idx];
          if (s2 >= 0.0f) {
            const float mh = p.c1 * l.z1[idx];
            const float vh = p.c2 * s2;
            const float den = p.eps + __builtin_amdgcn_sqrtf(vh);
            l.z1[idx] = p.lr * (mh * __builtin_amdgcn_rcpf(den));
            l.z2[idx] = -1.0f;
          }
        }
      };
      if (staged) {
        int row = 0, col = 0;
#pragma unroll
        for (int c = 0; c < kChunks; ++c) {
          if (row < n_old) add(stg[c], n_old - row);
          if (++col == R) { col = 0; ++row; }
        }
      } else {
        for (int i = 0, slot = slot0; i < n_old; ++i, slot = (slot + 1 == m) ? 0 : slot + 1)
          for (int jj = lane; jj < kq; jj += kWave) add(E::load(rw, slot * kq + jj), n_old - i);
      }
      for (int jj = lane; jj < kq; jj += kWave) add(E::lds_get(l.newrow, jj), 0);
      if (staged) {
#pragma unroll
        for (int c = 0; c < kChunks; ++c) convert(stg[c]);
      } else {
        for (int i = 0, slot = slot0; i < n_old; ++i, slot = (slot + 1 == m) ? 0 : slot + 1)
          for (int jj = lane; jj < kq; jj += kWave) convert(E::load(rw, slot * kq + jj));
      }
      for (int jj = lane; jj < kq; jj += kWave) convert(E::lds_get(l.newrow, jj));
    }

    // ---------------------------------------------- 3. e = Q(a with a[I] = 0)
    {
      const float Tf = __uint_as_float(T);
      const Rsrc re = make_rsrc(cur.ef, (((uint32_t)s + 1) / 2 + 3) & ~3u);
      const uint32_t nbk = ((uint32_t)s + (1u << bucket_log2) - 1) >> bucket_log2;
      const Rsrc rs = make_rsrc(cur.stats, nbk * 8);
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        const uint32_t i0 = v * NT * 8 + tid * 8;
        float x[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float ab = __builtin_fabsf(a[v][e]);
          const bool kept = notie ? (ab >= Tf) : (ab > Tf || (ab == Tf && i0 + e <= i_last));
          x[e] = kept ? 0.0f : a[v][e];
        }
        float mn, mx;
        if (full) {
          mn = __builtin_fminf(__builtin_fminf(__builtin_fminf(x[0], x[1]), x[2]),
                               __builtin_fminf(__builtin_fminf(x[3], x[4]), x[5]));
          mn = __builtin_fminf(mn, __builtin_fminf(x[6], x[7]));
          mx = __builtin_fmaxf(__builtin_fmaxf(__builtin_fmaxf(x[0], x[1]), x[2]),
                               __builtin_fmaxf(__builtin_fmaxf(x[3], x[4]), x[5]));
          mx = __builtin_fmaxf(mx, __builtin_fmaxf(x[6], x[7]));
        } else {
          mn = __builtin_inff();
          mx = -__builtin_inff();
#pragma unroll
          for (int e = 0; e < 8; ++e)
            if ((int)(i0 + e) < s) { mn = __builtin_fminf(mn, x[e]); mx = __builtin_fmaxf(mx, x[e]); }
        }
        group_minmax(mn, mx, G);
        mn = mn + 0.0f;  // a bucket bound of -0 is stored as +0
        mx = mx + 0.0f;
        const float u = div15(mx - mn);
        // Codes from two products that bracket the quotient: v_rcp is within
        // 1 ulp for these u, so r_lo < 1/u < r_hi and
        // rint((x-min)*r_lo) <= rint((x-min)/u) <= rint((x-min)*r_hi).  Where
        // the two agree (all but a few elements in a million) the code is
        // exact; elsewhere it is recomputed with an IEEE division.
        const float rcp = __builtin_amdgcn_rcpf(u);
        const float r_lo = __uint_as_float(__float_as_uint(rcp) - 2u);
        const float r_hi = __uint_as_float(__float_as_uint(rcp) + 2u);
        uint32_t d1e = 0, d1o = 0, d2e = 0, d2o = 0;
#pragma unroll
        for (int h = 0; h < 4; ++h) {
          const float ye = x[2 * h] - mn, yo = x[2 * h + 1] - mn;
          const float p1e = ye * r_lo, p1o = yo * r_lo;
          const float p2e = ye * r_hi, p2o = yo * r_hi;
          d1e = __builtin_amdgcn_cvt_pk_u8_f32(p1e, h, d1e);  // round half to even, clamp to [0, 255]
          d1o = __builtin_amdgcn_cvt_pk_u8_f32(p1o, h, d1o);
          d2e = __builtin_amdgcn_cvt_pk_u8_f32(p2e, h, d2e);
          d2o = __builtin_amdgcn_cvt_pk_u8_f32(p2o, h, d2o);
        }
        uint32_t w = d1e | (d1o << 4);
        const bool exact_u = u >= 0x1p-125f && u <= 0x1p+125f;
        if (!exact_u || d1e != d2e || d1o != d2o) {
          w = 0;
          if (u != 0.0f) {
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              const float y = x[e] - mn;
              float rr = __builtin_rintf(y / u);
              rr = __builtin_fminf(__builtin_fmaxf(rr, 0.0f), 15.0f);
              w |= (uint32_t)rr << (4 * e);
            }
          }
        }
        if (!full) {
#pragma unroll
          for (int e = 0; e < 8; ++e)
            if ((int)(i0 + e) >= s) w &= ~(0xFu << (4 * e));
        }
        if ((int)i0 < s) {
          __builtin_amdgcn_raw_buffer_store_b32(w, re, i0 >> 1, 0, 0);
          if ((i0 & ((1u << bucket_log2) - 1)) == 0)
            __builtin_amdgcn_raw_buffer_store_b64(u32x2{__float_as_uint(mn), __float_as_uint(mx)}, rs,
                                                  (i0 >> bucket_log2) * 8, 0, 0);
        }
      }
    }
    lds_sync();  // B4 ------------------------------------------------

    // ---------------------------------------------- 6. parameter update
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      const uint32_t i0 = v * NT * 8 + tid * 8;
      if ((int)i0 >= s) continue;
      const float4 u0 = *(const float4*)(l.z1 + i0);
      const float4 u1 = *(const float4*)(l.z1 + i0 + 4);
      const float upd[8] = {u0.x, u0.y, u0.z, u0.w, u1.x, u1.y, u1.z, u1.w};
      // leave the moments cleared for the next block (only this thread reads
      // these entries from here on)
      const float4 zero = make_float4(0.f, 0.f, 0.f, 0.f);
      *(float4*)(l.z1 + i0) = zero;
      *(float4*)(l.z1 + i0 + 4) = zero;
      *(float4*)(l.z2 + i0) = zero;
      *(float4*)(l.z2 + i0 + 4) = zero;
      float thf[8], out[8];
      unpack8<PBF16>(th[v], thf);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float base = p.decay_is_one ? thf[e] : thf[e] * p.decay;
        out[e] = base - upd[e];
      }
      store8<PBF16>(rp, i0, s, full, out);
    }

    if (!has_next) break;
    pre = npre;
    ++gb;
  }
}

// The bf16 parameter / bf16 gradient / bf16 window variant (the paper's
// training setting) is held to 128 VGPRs for four waves per SIMD; the
// float32 variants keep their natural register budget.
template <int NT, bool PBF16, bool GBF16, bool VF32>
__global__ void __launch_bounds__(NT) step_kernel(StepParams p) {
  step_body<NT, PBF16, GBF16, VF32>(p);
}

template <int NT>
__global__ void __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(4))) step_kernel_bf16(StepParams p) {
  step_body<NT, true, true, false>(p);
}

// ================================================== debug: dense moments
// One workgroup per block of one tensor: rebuild z1, z2 from every live row
// (oldest first) and write m-hat = c1 z1, v-hat = c2 z2.
template <int NT, bool VF32>
__global__ void __launch_bounds__(NT) moments_kernel(StepParams p, int32_t tensor,
                                                     int64_t first_block, float* mhat,
                                                     float* vhat) {
  constexpr int CAP = NT * 16;
  using E = Entry<VF32>;
  extern __shared__ __align__(16) uint32_t smem[];
  float* z1 = (float*)smem;
  float* z2 = z1 + CAP;
  const TensorDesc d = p.tensors[tensor];
  const int64_t q = (int64_t)blockIdx.x + first_block - d.first_block;
  const int64_t e0 = q * p.block;
  const int s = (int)((d.numel - e0 < p.block) ? (d.numel - e0) : p.block);
  const int kq = (q == d.num_blocks - 1) ? d.k_last : d.k_full;
  const Rsrc rw = make_rsrc(p.state + d.win_off + (uint64_t)q * p.window * d.k_full * E::kWords * 4,
                            (uint32_t)(p.window * kq * E::kWords * 4));
  for (int x = threadIdx.x; x < CAP; x += NT) { z1[x] = 0.0f; z2[x] = 0.0f; }
  __syncthreads();
  if (threadIdx.x < kWave) {
    const int n_live = p.n_old + 1;
    for (int o = 0; o < n_live; ++o) {
      const int64_t sstep = p.t - n_live + 1 + o;
      const int slot = (int)((sstep - 1) % p.window);
      const int r = (int)(p.t - sstep);
      for (int jj = threadIdx.x; jj < kq; jj += kWave) {
        const typename E::T e = E::load(rw, slot * kq + jj);
        const uint32_t idx = E::idx(e);
        if (idx < (uint32_t)s) {
          const float v = E::val(e);
          const float x1 = p.wpow[r] * v;
          const float vv = v * v;
          const float x2 = p.wpow[kMaxWindow + r] * vv;
          z1[idx] = z1[idx] + x1;
          z2[idx] = z2[idx] + x2;
        }
      }
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < s; i += NT) {
    mhat[e0 + i] = p.c1 * z1[i];
    vhat[e0 + i] = p.c2 * z2[i];
  }
}

template <int NT, bool PB, bool GB, bool VF>
hipError_t launch_one(const StepParams& p, hipStream_t stream) {
  auto kern = (PB && GB && !VF) ? step_kernel_bf16<NT> : step_kernel<NT, PB, GB, VF>;
  const size_t lds = lds_words<NT>(p.k_full, VF ? 2 : 1) * 4;
  // one persistent workgroup per resident slot of the device
  static int slots = -1, cus = -1;
  static size_t slots_lds = 0;
  if (slots < 0 || slots_lds != lds) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
    if (e == hipSuccess)
      e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&slots, reinterpret_cast<const void*>(kern), NT, lds);
    if (e != hipSuccess) return e;
    if (slots < 1) slots = 1;
    slots_lds = lds;
  }
  int64_t grid = (int64_t)slots * cus;
  if (grid > p.total_blocks) grid = p.total_blocks;
  hipLaunchKernelGGL(kern, dim3((uint32_t)grid), dim3(NT), lds, stream, p);
  return hipGetLastError();
}

template <int NT>
hipError_t launch_dtypes(const StepParams& p, int pb, int gb, int vf, hipStream_t stream) {
  const int sel = (pb ? 4 : 0) | (gb ? 2 : 0) | (vf ? 1 : 0);
  switch (sel) {
    case 0: return launch_one<NT, false, false, false>(p, stream);
    case 1: return launch_one<NT, false, false, true>(p, stream);
    case 2: return launch_one<NT, false, true, false>(p, stream);
    case 3: return launch_one<NT, false, true, true>(p, stream);
    case 4: return launch_one<NT, true, false, false>(p, stream);
    case 5: return launch_one<NT, true, false, true>(p, stream);
    case 6: return launch_one<NT, true, true, false>(p, stream);
    default: return launch_one<NT, true, true, true>(p, stream);
  }
}

}  // namespace

size_t step_lds_bytes(int block, int k_full, int value_f32) {
  const int ew = value_f32 ? 2 : 1;
  return (threads_for_block(block) == 64 ? lds_words<64>(k_full, ew) : lds_words<256>(k_full, ew)) * 4;
}

hipError_t launch_step(const StepParams& p, int param_bf16, int grad_bf16, int value_f32,
                       hipStream_t stream) {
  if (threads_for_block(p.block) == 64) return launch_dtypes<64>(p, param_bf16, grad_bf16, value_f32, stream);
  return launch_dtypes<256>(p, param_bf16, grad_bf16, value_f32, stream);
}

hipError_t launch_moments(const StepParams& p, int32_t tensor, int64_t first_block, int64_t grid,
                          float* mhat, float* vhat, int value_f32, hipStream_t stream) {
  const int nt = threads_for_block(p.block);
  const size_t lds = (size_t)2 * nt * 16 * 4;
  if (nt == 64) {
    if (value_f32)
      hipLaunchKernelGGL((moments_kernel<64, true>), dim3((uint32_t)grid), dim3(64), lds, stream, p, tensor,
                         first_block, mhat, vhat);
    else
      hipLaunchKernelGGL((moments_kernel<64, false>), dim3((uint32_t)grid), dim3(64), lds, stream, p, tensor,
                         first_block, mhat, vhat);
  } else {
    if (value_f32)
      hipLaunchKernelGGL((moments_kernel<256, true>), dim3((uint32_t)grid), dim3(256), lds, stream, p, tensor,
                         first_block, mhat, vhat);
    else
      hipLaunchKernelGGL((moments_kernel<256, false>), dim3((uint32_t)grid), dim3(256), lds, stream, p,
                         tensor, first_block, mhat, vhat);
  }
  return hipGetLastError();
}

}  // namespace microadam
