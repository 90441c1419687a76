// MicroAdam step kernels for CDNA4 (gfx950).
//
// One workgroup owns one Top-K block of B_d elements of one tensor and runs
// the whole step of Algorithm 1 for it in a single pass over HBM:
//   1. load the block's gradient, parameters, 4-bit EF codes, bucket
//      (delta, Delta) pairs and the older window rows (all loads issued first);
//   2. a = g + Q^-1(e)                           (Algorithm 1, Algorithm 2 Q^-1)
//   3. block Top-K of |a|, lower index wins ties  (Section 3.1, "Top-K")
//   4. a[I] = 0, bucket min/max by lane shuffles, e = Q(a) packed two codes
//      per byte                                   (Algorithm 1; Section 3.1)
//   5. the new window row (I, bf16(V)) is stored  (Section 3.2 layout)
//   6. m-hat, v-hat rebuilt from the window in LDS, weights beta^(t-s)
//                                                  (Algorithm 2, AdamStats)
//   7. theta <- (1 - eta*lambda) theta - eta m / (eps + sqrt(v))
//                                                  (Algorithm 1, Algorithm 4)
// Nothing crosses blocks, so no workgroup talks to another.
//
// Element layout inside a block: thread `tid` of NT owns NV = EPT/8 vectors of
// 8 consecutive elements; vector v holds elements v*NT*8 + tid*8 + [0, 8).
// Every wave-wide load or store instruction therefore covers one contiguous
// span (1 KiB of bf16 per wave), and an EF bucket of B_q elements is held by
// B_q/8 neighbouring lanes.
//
// Arithmetic that decides an integer (EF decode, accumulator, Top-K keys,
// bucket min/max, codes) is binary32 with one rounding per operation: this
// file is compiled with -ffp-contract=off and the divisions are IEEE.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "microadam_device.h"

namespace microadam {
namespace {

constexpr int kWave = 64;
constexpr float kLevels = 15.0f;   // 2^b - 1 for b = 4

// ---------------------------------------------------------------- wave ops
__device__ __forceinline__ uint64_t ballot(bool p) { return __ballot(p); }

__device__ __forceinline__ uint32_t lanes_below(uint64_t m) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                   __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
}

__device__ __forceinline__ uint32_t popc(uint64_t m) { return (uint32_t)__popcll(m); }

__device__ __forceinline__ uint32_t uniform(uint32_t x) {
  return __builtin_amdgcn_readfirstlane(x);
}

template <int CTRL>
__device__ __forceinline__ float dpp_mov(float x) {
  return __builtin_bit_cast(
      float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xF, 0xF, false));
}

// min / max over groups of G neighbouring lanes (G a power of two <= 64).
__device__ __forceinline__ void group_minmax(float& mn, float& mx, int G) {
  if (G > 1) {  // partner lane ^ 1
    mn = fminf(mn, dpp_mov<0xB1>(mn));
    mx = fmaxf(mx, dpp_mov<0xB1>(mx));
  }
  if (G > 2) {  // partner lane ^ 2
    mn = fminf(mn, dpp_mov<0x4E>(mn));
    mx = fmaxf(mx, dpp_mov<0x4E>(mx));
  }
  if (G > 4) {  // mirror within 8 lanes: pairs the two uniform quads
    mn = fminf(mn, dpp_mov<0x141>(mn));
    mx = fmaxf(mx, dpp_mov<0x141>(mx));
  }
  if (G > 8) {  // mirror within 16 lanes: pairs the two uniform 8-groups
    mn = fminf(mn, dpp_mov<0x140>(mn));
    mx = fmaxf(mx, dpp_mov<0x140>(mx));
  }
  for (int off = 16; off < G; off <<= 1) {
    mn = fminf(mn, __shfl_xor(mn, off, kWave));
    mx = fmaxf(mx, __shfl_xor(mx, off, kWave));
  }
}

// ------------------------------------------------------------ element I/O
__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

__device__ __forceinline__ uint32_t to_bf16_bits(float x) {
  __bf16 b = (__bf16)x;  // v_cvt_pk_bf16_f32: round half to even
  return (uint32_t)__builtin_bit_cast(uint16_t, b);
}

// Loads 8 consecutive elements starting at element `base` of `p`; elements
// at or after `limit` read as 0.  `full` = all 8 are below limit.
template <bool BF16>
__device__ __forceinline__ void load8(const void* p, int64_t base, int64_t limit, float out[8]) {
  if (BF16) {
    const uint16_t* q = (const uint16_t*)p + base;
    if (base + 8 <= limit) {
      uint4 w = *(const uint4*)q;
      out[0] = bf16_lo(w.x); out[1] = bf16_hi(w.x);
      out[2] = bf16_lo(w.y); out[3] = bf16_hi(w.y);
      out[4] = bf16_lo(w.z); out[5] = bf16_hi(w.z);
      out[6] = bf16_lo(w.w); out[7] = bf16_hi(w.w);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        out[e] = (base + e < limit) ? __uint_as_float((uint32_t)q[e] << 16) : 0.0f;
    }
  } else {
    const float* q = (const float*)p + base;
    if (base + 8 <= limit) {
      float4 x0 = *(const float4*)q, x1 = *(const float4*)(q + 4);
      out[0] = x0.x; out[1] = x0.y; out[2] = x0.z; out[3] = x0.w;
      out[4] = x1.x; out[5] = x1.y; out[6] = x1.z; out[7] = x1.w;
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) out[e] = (base + e < limit) ? q[e] : 0.0f;
    }
  }
}

template <bool BF16>
__device__ __forceinline__ void store8(void* p, int64_t base, int64_t limit, const float in[8]) {
  if (BF16) {
    uint16_t* q = (uint16_t*)p + base;
    if (base + 8 <= limit) {
      uint4 w;
      w.x = to_bf16_bits(in[0]) | (to_bf16_bits(in[1]) << 16);
      w.y = to_bf16_bits(in[2]) | (to_bf16_bits(in[3]) << 16);
      w.z = to_bf16_bits(in[4]) | (to_bf16_bits(in[5]) << 16);
      w.w = to_bf16_bits(in[6]) | (to_bf16_bits(in[7]) << 16);
      *(uint4*)q = w;
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (base + e < limit) q[e] = (uint16_t)to_bf16_bits(in[e]);
    }
  } else {
    float* q = (float*)p + base;
    if (base + 8 <= limit) {
      *(float4*)q = make_float4(in[0], in[1], in[2], in[3]);
      *(float4*)(q + 4) = make_float4(in[4], in[5], in[6], in[7]);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e)
        if (base + e < limit) q[e] = in[e];
    }
  }
}

// ------------------------------------------------------- window entries
// bf16 values: one word (index | bf16 << 16); f32 values: (index, value).
template <bool VF32>
struct Entry {
  static constexpr int kWords = VF32 ? 2 : 1;
  __device__ static void put(uint32_t* dst, uint32_t idx, float v) {
    if (VF32) { dst[0] = idx; dst[1] = __float_as_uint(v); }
    else dst[0] = idx | (to_bf16_bits(v) << 16);
  }
  __device__ static void get(const uint32_t* src, uint32_t& idx, float& v) {
    if (VF32) { idx = src[0]; v = __uint_as_float(src[1]); }
    else { uint32_t w = src[0]; idx = w & 0xFFFFu; v = __uint_as_float(w & 0xFFFF0000u); }
  }
};

// LDS carve-up (in 32-bit words), shared by the step and moment kernels.
struct Lds {
  float* z1;            // capacity floats: sum of beta1^r V, later the update
  float* z2;            // capacity floats: sum of beta2^r V^2
  uint32_t* cand_bits;  // kCandCap candidate values (float bits)
  uint32_t* cand_idx;   // kCandCap candidate block-relative indices
  uint32_t* red;        // 4 x 64 words of reduction scratch
  uint32_t* bcast;      // 8 broadcast words
  uint32_t* newrow;     // k_full entries of the row written at step t
  uint32_t* stage;      // staged older rows (stage_slots * k_q entries)
};

__device__ __forceinline__ Lds carve(uint32_t* smem, int capacity, int k_full, int words) {
  Lds l;
  l.z1 = (float*)smem;
  l.z2 = l.z1 + capacity;
  l.cand_bits = (uint32_t*)(l.z2 + capacity);
  l.cand_idx = l.cand_bits + kCandCap;
  l.red = l.cand_idx + kCandCap;
  l.bcast = l.red + 4 * 64;
  l.newrow = l.bcast + 8;
  l.stage = l.newrow + k_full * words;
  return l;
}

enum { B_T = 0, B_ILAST = 1, B_L = 2 };

// Exclusive prefix, in element order, of per-(thread, vector) counts < 16.
// Returns the workgroup total; base[v] = number of counted elements that come
// before this thread's vector v.  `red` needs NV*NW words.  Contains one barrier;
// `red` must not be reused until a later barrier.
template <int NT, int NV>
__device__ __forceinline__ uint32_t wg_scan(const uint32_t (&cnt)[NV], uint32_t (&base)[NV],
                                            uint32_t* red) {
  constexpr int NW = NT / kWave;
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  uint32_t pre[NV];
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    const uint64_t b0 = ballot(cnt[v] & 1u), b1 = ballot(cnt[v] & 2u);
    const uint64_t b2 = ballot(cnt[v] & 4u), b3 = ballot(cnt[v] & 8u);
    pre[v] = lanes_below(b0) + 2u * lanes_below(b1) + 4u * lanes_below(b2) + 8u * lanes_below(b3);
    const uint32_t tot = popc(b0) + 2u * popc(b1) + 4u * popc(b2) + 8u * popc(b3);
    if (lane == 0) red[v * NW + wave] = tot;
  }
  __syncthreads();
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

// Workgroup-wide count of a per-element predicate given as NV 8-bit masks.
// One barrier; `red` (NW words) must differ between consecutive calls.
template <int NT, int NV>
__device__ __forceinline__ uint32_t wg_count(const uint32_t (&mask)[NV], uint32_t* red) {
  constexpr int NW = NT / kWave;
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  uint32_t c = 0;
#pragma unroll
  for (int v = 0; v < NV; ++v) c += __popc(mask[v]);
  // wave sum of small per-lane counts (<= 8*NV) by bit slices
  constexpr int kBits = (NV <= 1) ? 4 : (NV <= 3) ? 5 : (NV <= 7) ? 6 : 7;
  uint32_t tot = 0;
#pragma unroll
  for (int b = 0; b < kBits; ++b) tot += popc(ballot((c >> b) & 1u)) << b;
  if (lane == 0) red[wave] = tot;
  __syncthreads();
  uint32_t s = 0;
#pragma unroll
  for (int w = 0; w < NW; ++w) s += red[w];
  return s;
}

// ------------------------------------------------- window rebuild (wave 0)
// Adds the rows of one block into z1/z2 in order, oldest first:
// z1[idx] += beta1^r V, z2[idx] += beta2^r V^2 (Algorithm 2).  Run by one
// wave; within a row the indices are distinct, so a row chunk of 64 entries
// has no conflicting lanes, and rows follow each other in program order.
// Indices at or above `s` (possible only in a corrupted restored state) are
// skipped so that LDS is never addressed outside the block.
template <bool VF32>
__device__ __forceinline__ void add_row(const Lds& l, const uint32_t* row, int kq, float w1,
                                        float w2, int lane, int s) {
  for (int j = lane; j < kq; j += kWave) {
    uint32_t idx;
    float v;
    Entry<VF32>::get(row + j * Entry<VF32>::kWords, idx, v);
    if (idx >= (uint32_t)s) continue;
    const float a = w1 * v;
    const float sq = v * v;
    const float b = w2 * sq;
    l.z1[idx] = l.z1[idx] + a;
    l.z2[idx] = l.z2[idx] + b;
  }
}

// Converts the moments at the row's indices into the parameter decrement
// eta * m / (eps + sqrt(v)), stored in z1; z2 = -1 marks an index already
// converted (a later row holding the same index skips it).
template <bool VF32>
__device__ __forceinline__ void convert_row(const Lds& l, const uint32_t* row, int kq,
                                            const StepParams& p, int lane, int s) {
  for (int j = lane; j < kq; j += kWave) {
    uint32_t idx;
    float v;
    Entry<VF32>::get(row + j * Entry<VF32>::kWords, idx, v);
    if (idx >= (uint32_t)s) continue;
    const float s2 = l.z2[idx];
    if (s2 >= 0.0f) {
      const float m = p.c1 * l.z1[idx];
      const float vv = p.c2 * s2;
      const float den = p.eps + sqrtf(vv);
      const float q = m / den;
      l.z1[idx] = p.lr * q;
      l.z2[idx] = -1.0f;
    }
  }
}

__device__ __forceinline__ void zero_lds(float* z, int n) {
  for (int x = threadIdx.x * 4; x < n; x += blockDim.x * 4)
    *(float4*)(z + x) = make_float4(0.f, 0.f, 0.f, 0.f);
}

// =================================================================== step
template <int NT, int EPT, bool PBF16, bool GBF16, bool VF32>
__global__ void __launch_bounds__(NT) step_kernel(StepParams p) {
  constexpr int NV = EPT / 8;
  constexpr int NW = NT / kWave;
  constexpr int CAP = NT * EPT;  // block capacity
  constexpr int EW = Entry<VF32>::kWords;
  extern __shared__ __align__(16) uint32_t smem[];
  const Lds l = carve(smem, CAP, p.k_full, EW);

  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const uint32_t gblock = blockIdx.x;
  const uint32_t tj = p.block_tensor[gblock];
  const TensorDesc d = p.tensors[tj];
  const int64_t q = (int64_t)gblock - d.first_block;
  const int64_t e0 = q * p.block;                                  // first element
  const int s = (int)((d.numel - e0 < p.block) ? (d.numel - e0) : p.block);  // valid
  const int kq = (q == d.num_blocks - 1) ? d.k_last : d.k_full;
  const int bucket_log2 = p.bucket_log2;

  uint8_t* const ef = p.state + d.ef_off + (e0 >> 1);
  float2* const stats = (float2*)(p.state + d.stats_off) + (e0 >> bucket_log2);
  uint32_t* const win = (uint32_t*)(p.state + d.win_off) + q * (int64_t)p.window * d.k_full * EW;

  // ---- 1. issue every load of the block
  float2 st[NV];
  uint32_t code_w[NV];
  float a[NV][8], th[NV][8];
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    const int i0 = v * NT * 8 + tid * 8;
    if (i0 < s) {
      st[v] = stats[i0 >> bucket_log2];
      code_w[v] = *(const uint32_t*)(ef + (i0 >> 1));
    } else {
      st[v] = make_float2(0.f, 0.f);
      code_w[v] = 0u;
    }
  }
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    const int i0 = v * NT * 8 + tid * 8;
    if (i0 < s) load8<GBF16>(d.grad, e0 + i0, d.numel, a[v]);
    else {
#pragma unroll
      for (int e = 0; e < 8; ++e) a[v][e] = 0.0f;
    }
  }
  // older window rows of this block, staged through registers into LDS
  const int stage_words = p.stage_slots * kq * EW;
  uint32_t stg[kStageSlots];
#pragma unroll
  for (int j = 0; j < kStageSlots; ++j) {
    const int x = tid + j * NT;
    stg[j] = (x < stage_words) ? win[x] : 0u;
  }
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    const int i0 = v * NT * 8 + tid * 8;
    if (i0 < s) load8<PBF16>(d.param, e0 + i0, d.numel, th[v]);
    else {
#pragma unroll
      for (int e = 0; e < 8; ++e) th[v][e] = 0.0f;
    }
  }
  zero_lds(l.z1, p.block);
  zero_lds(l.z2, p.block);

  // ---- 2. accumulator a = g + Q^-1(e): x_Q * u + delta, u = (Delta - delta)/15
  uint32_t key[NV][8];
  uint32_t valid[NV];  // 8-bit masks
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    const int i0 = v * NT * 8 + tid * 8;
    const float lo = st[v].x, hi = st[v].y;
    const float u = (hi - lo) / kLevels;
    valid[v] = 0u;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float c = (float)((code_w[v] >> (4 * e)) & 15u);
      const float scaled = c * u;
      const float dec = scaled + lo;
      a[v][e] = a[v][e] + dec;
      const bool ok = i0 + e < s;
      valid[v] |= (ok ? 1u : 0u) << e;
      key[v][e] = ok ? (__float_as_uint(a[v][e]) & 0x7FFFFFFFu) : 0u;
    }
  }

  // ---- 3. block Top-K of |a|: threshold key T and the last index i_last
  //         among keys equal to T, so element i is kept iff
  //         key > T or (key == T and i <= i_last).
  uint32_t T, i_last;
  {
    // Fast path: a lower bound L on the k-th largest key from the per-wave
    // ceil(k/NW)-th largest lane maximum; the few keys >= L are resolved
    // exactly by wave 0.
    uint32_t lmax = 0;
#pragma unroll
    for (int v = 0; v < NV; ++v)
#pragma unroll
      for (int e = 0; e < 8; ++e) lmax = max(lmax, key[v][e]);
    const int kw = (kq + NW - 1) / NW;
    bool fast = kq <= kWave * NW;
    uint32_t L = 0;
    if (fast) {
      uint32_t P = 0;
      for (int b = 30; b >= 0; --b) {
        const uint32_t c = P | (1u << b);
        if ((int)popc(ballot(lmax >= c)) >= kw) P = c;
      }
      if (lane == 0) l.red[3 * 64 + wave] = P;
      __syncthreads();
      L = l.red[3 * 64];
#pragma unroll
      for (int w = 1; w < NW; ++w) L = min(L, l.red[3 * 64 + w]);
    }
    uint32_t cnt[NV], base[NV];
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      uint32_t c = 0;
#pragma unroll
      for (int e = 0; e < 8; ++e) c += ((valid[v] >> e) & 1u) && key[v][e] >= L;
      cnt[v] = c;
    }
    // Consecutive scans / counts alternate between two reduction buffers:
    // a buffer is rewritten only after the barrier of the call in between.
    int buf = 0;
    const uint32_t C = fast ? wg_scan<NT, NV>(cnt, base, l.red) : 0u;
    if (fast) buf = 1;
    fast = fast && C <= (uint32_t)kCandCap;
    if (fast) {
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        uint32_t pos = base[v];
        const int i0 = v * NT * 8 + tid * 8;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          if (((valid[v] >> e) & 1u) && key[v][e] >= L) {
            l.cand_bits[pos] = __float_as_uint(a[v][e]);
            l.cand_idx[pos] = (uint32_t)(i0 + e);
            ++pos;
          }
        }
      }
      __syncthreads();
      if (wave == 0) {
        uint32_t ck[4], cb[4], ci[4];
        bool cv[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const uint32_t j = lane + kWave * r;
          cv[r] = j < C;
          cb[r] = cv[r] ? l.cand_bits[j] : 0u;
          ci[r] = cv[r] ? l.cand_idx[j] : 0u;
          ck[r] = cb[r] & 0x7FFFFFFFu;
        }
        uint32_t Tw = 0;
        for (int b = 30; b >= 0; --b) {
          const uint32_t c = Tw | (1u << b);
          uint32_t n = 0;
#pragma unroll
          for (int r = 0; r < 4; ++r) n += popc(ballot(cv[r] && ck[r] >= c));
          if ((int)n >= kq) Tw = c;
        }
        uint32_t ngt = 0;
#pragma unroll
        for (int r = 0; r < 4; ++r) ngt += popc(ballot(cv[r] && ck[r] > Tw));
        const uint32_t need = (uint32_t)kq - ngt;  // >= 1
        uint32_t eq_before = 0, sel_before = 0;
        uint32_t* row = win + (int64_t)p.new_slot * kq * EW;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const bool gt = cv[r] && ck[r] > Tw;
          const bool eq = cv[r] && ck[r] == Tw;
          const uint64_t eqm = ballot(eq);
          const uint32_t rank = eq_before + lanes_below(eqm);
          eq_before += popc(eqm);
          if (eq && rank == need - 1) l.bcast[B_ILAST] = ci[r];
          const bool sel = gt || (eq && rank < need);
          const uint64_t sm = ballot(sel);
          const uint32_t pos = sel_before + lanes_below(sm);
          sel_before += popc(sm);
          if (sel) {
            Entry<VF32>::put(row + pos * EW, ci[r], __uint_as_float(cb[r]));
            Entry<VF32>::put(l.newrow + pos * EW, ci[r], __uint_as_float(cb[r]));
          }
        }
        if (lane == 0) l.bcast[B_T] = Tw;
      }
      __syncthreads();
      T = l.bcast[B_T];
      i_last = l.bcast[B_ILAST];
    } else {
      // General path: bitwise search for the k-th largest key over the block.
      uint32_t P = 0;
      for (int b = 30; b >= 0; --b) {
        const uint32_t c = P | (1u << b);
        uint32_t m[NV];
#pragma unroll
        for (int v = 0; v < NV; ++v) {
          uint32_t x = 0;
#pragma unroll
          for (int e = 0; e < 8; ++e) x |= (uint32_t)(((valid[v] >> e) & 1u) && key[v][e] >= c) << e;
          m[v] = x;
        }
        const uint32_t n = wg_count<NT, NV>(m, l.red + 64 * buf);
        buf ^= 1;
        if ((int)n >= kq) P = c;
      }
      T = P;
      uint32_t gtm[NV], eqm[NV];
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        uint32_t g = 0, q2 = 0;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const bool ok = (valid[v] >> e) & 1u;
          g |= (uint32_t)(ok && key[v][e] > T) << e;
          q2 |= (uint32_t)(ok && key[v][e] == T) << e;
        }
        gtm[v] = g;
        eqm[v] = q2;
      }
      const uint32_t ngt = wg_count<NT, NV>(gtm, l.red + 64 * buf);
      buf ^= 1;
      const uint32_t need = (uint32_t)kq - ngt;
      uint32_t ecnt[NV], ebase[NV];
#pragma unroll
      for (int v = 0; v < NV; ++v) ecnt[v] = __popc(eqm[v]);
      (void)wg_scan<NT, NV>(ecnt, ebase, l.red + 64 * buf);
      buf ^= 1;
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        const int i0 = v * NT * 8 + tid * 8;
        uint32_t r = ebase[v];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          if ((eqm[v] >> e) & 1u) {
            if (r == need - 1) l.bcast[B_ILAST] = (uint32_t)(i0 + e);
            ++r;
          }
        }
      }
      __syncthreads();
      i_last = l.bcast[B_ILAST];
      // compact the kept entries, in index order, into the new window row
      uint32_t scnt[NV], sbase[NV];
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        const int i0 = v * NT * 8 + tid * 8;
        uint32_t c = 0;
#pragma unroll
        for (int e = 0; e < 8; ++e)
          c += ((gtm[v] >> e) & 1u) || (((eqm[v] >> e) & 1u) && (uint32_t)(i0 + e) <= i_last);
        scnt[v] = c;
      }
      (void)wg_scan<NT, NV>(scnt, sbase, l.red + 64 * buf);
      uint32_t* row = win + (int64_t)p.new_slot * kq * EW;
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        const int i0 = v * NT * 8 + tid * 8;
        uint32_t pos = sbase[v];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const bool sel = ((gtm[v] >> e) & 1u) || (((eqm[v] >> e) & 1u) && (uint32_t)(i0 + e) <= i_last);
          if (sel) {
            Entry<VF32>::put(row + pos * EW, (uint32_t)(i0 + e), a[v][e]);
            Entry<VF32>::put(l.newrow + pos * EW, (uint32_t)(i0 + e), a[v][e]);
            ++pos;
          }
        }
      }
    }
  }

  // older rows into LDS (made visible by the barrier below)
#pragma unroll
  for (int j = 0; j < kStageSlots; ++j) {
    const int x = tid + j * NT;
    if (x < stage_words) l.stage[x] = stg[j];
  }
  __syncthreads();

  // ---- 6. wave 0 rebuilds the moments while the other waves quantize
  if (wave == 0) {
    const int64_t t = p.t;
    for (int o = 0; o < p.n_old; ++o) {
      const int64_t sstep = t - p.n_old + o;           // step that wrote the row
      const int slot = (int)((sstep - 1) % p.window);
      const int r = (int)(t - sstep);
      const uint32_t* row = p.stage_slots ? l.stage + slot * kq * EW
                                          : win + (int64_t)slot * kq * EW;
      add_row<VF32>(l, row, kq, p.w1[r], p.w2[r], lane, s);
    }
    add_row<VF32>(l, l.newrow, kq, p.w1[0], p.w2[0], lane, s);
    for (int o = 0; o < p.n_old; ++o) {
      const int64_t sstep = t - p.n_old + o;
      const int slot = (int)((sstep - 1) % p.window);
      const uint32_t* row = p.stage_slots ? l.stage + slot * kq * EW
                                          : win + (int64_t)slot * kq * EW;
      convert_row<VF32>(l, row, kq, p, lane, s);
    }
    convert_row<VF32>(l, l.newrow, kq, p, lane, s);
  }

  // ---- 4. a[I] = 0; bucket (delta, Delta) = (min, max); e = Q(a)
  const int G = (1 << bucket_log2) >> 3;  // lanes per bucket
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    const int i0 = v * NT * 8 + tid * 8;
    float mn = __builtin_inff(), mx = -__builtin_inff();
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const uint32_t i = (uint32_t)(i0 + e);
      const bool kept = key[v][e] > T || (key[v][e] == T && i <= i_last);
      const bool ok = (valid[v] >> e) & 1u;
      const float x = (ok && kept) ? 0.0f : a[v][e];
      a[v][e] = x;
      if (ok) {
        mn = fminf(mn, x);
        mx = fmaxf(mx, x);
      }
    }
    group_minmax(mn, mx, G);
    mn = mn + 0.0f;  // -0 is stored as +0
    mx = mx + 0.0f;
    const float u = (mx - mn) / kLevels;
    uint32_t w = 0;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      uint32_t c = 0;
      if (u != 0.0f) {
        const float y = (a[v][e] - mn) / u;
        float r = rintf(y);
        r = fminf(fmaxf(r, 0.0f), kLevels);
        c = (uint32_t)r;
      }
      c = ((valid[v] >> e) & 1u) ? c : 0u;
      w |= c << (4 * e);
    }
    if (i0 < s) {
      *(uint32_t*)(ef + (i0 >> 1)) = w;
      if ((i0 & ((1 << bucket_log2) - 1)) == 0) stats[i0 >> bucket_log2] = make_float2(mn, mx);
    }
  }
  __syncthreads();

  // ---- 7. theta <- theta * (1 - eta*lambda) - eta * m / (eps + sqrt(v))
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    const int i0 = v * NT * 8 + tid * 8;
    if (i0 >= s) continue;
    const float4 u0 = *(const float4*)(l.z1 + i0);
    const float4 u1 = *(const float4*)(l.z1 + i0 + 4);
    const float upd[8] = {u0.x, u0.y, u0.z, u0.w, u1.x, u1.y, u1.z, u1.w};
    float out[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float base = p.decay_is_one ? th[v][e] : th[v][e] * p.decay;
      out[e] = base - upd[e];
    }
    store8<PBF16>(d.param, e0 + i0, d.numel, out);
  }
}

// ================================================== debug: dense moments
template <int NT, bool VF32>
__global__ void __launch_bounds__(NT) moments_kernel(StepParams p, int32_t tensor,
                                                     int64_t first_block, float* mhat,
                                                     float* vhat) {
  constexpr int CAP = NT * 16;
  constexpr int EW = Entry<VF32>::kWords;
  extern __shared__ __align__(16) uint32_t smem[];
  const Lds l = carve(smem, CAP, p.k_full, EW);
  const TensorDesc d = p.tensors[tensor];
  const int64_t q = (int64_t)blockIdx.x + first_block - d.first_block;
  const int64_t e0 = q * p.block;
  const int s = (int)((d.numel - e0 < p.block) ? (d.numel - e0) : p.block);
  const int kq = (q == d.num_blocks - 1) ? d.k_last : d.k_full;
  const uint32_t* win = (const uint32_t*)(p.state + d.win_off) + q * (int64_t)p.window * d.k_full * EW;
  zero_lds(l.z1, p.block);
  zero_lds(l.z2, p.block);
  __syncthreads();
  if (threadIdx.x < kWave) {
    const int n_live = p.n_old + 1;  // rows written up to and including step t
    for (int o = 0; o < n_live; ++o) {
      const int64_t sstep = p.t - n_live + 1 + o;
      const int slot = (int)((sstep - 1) % p.window);
      const int r = (int)(p.t - sstep);
      add_row<VF32>(l, win + (int64_t)slot * kq * EW, kq, p.w1[r], p.w2[r], threadIdx.x, s);
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < s; i += NT) {
    mhat[e0 + i] = p.c1 * l.z1[i];
    vhat[e0 + i] = p.c2 * l.z2[i];
  }
}

template <int NT, int EPT, bool PB, bool GB, bool VF>
hipError_t launch_one(const StepParams& p, int64_t grid, size_t lds, hipStream_t stream) {
  hipLaunchKernelGGL((step_kernel<NT, EPT, PB, GB, VF>), dim3((uint32_t)grid), dim3(NT), lds,
                     stream, p);
  return hipGetLastError();
}

template <int NT, int EPT>
hipError_t launch_dtypes(const StepParams& p, int64_t grid, size_t lds, int pb, int gb, int vf,
                         hipStream_t stream) {
  const int sel = (pb ? 4 : 0) | (gb ? 2 : 0) | (vf ? 1 : 0);
  switch (sel) {
    case 0: return launch_one<NT, EPT, false, false, false>(p, grid, lds, stream);
    case 1: return launch_one<NT, EPT, false, false, true>(p, grid, lds, stream);
    case 2: return launch_one<NT, EPT, false, true, false>(p, grid, lds, stream);
    case 3: return launch_one<NT, EPT, false, true, true>(p, grid, lds, stream);
    case 4: return launch_one<NT, EPT, true, false, false>(p, grid, lds, stream);
    case 5: return launch_one<NT, EPT, true, false, true>(p, grid, lds, stream);
    case 6: return launch_one<NT, EPT, true, true, false>(p, grid, lds, stream);
    default: return launch_one<NT, EPT, true, true, true>(p, grid, lds, stream);
  }
}

}  // namespace

size_t step_lds_bytes(const StepParams& p, int value_f32) {
  const int nt = threads_for_block(p.block);
  const int cap = nt * 16;
  const int ew = value_f32 ? 2 : 1;
  size_t words = 2 * (size_t)cap + 2 * kCandCap + 4 * 64 + 8 + (size_t)p.k_full * ew +
                 (size_t)p.stage_slots * p.k_full * ew;
  return words * 4;
}

hipError_t launch_step(const StepParams& p, int64_t grid, int param_bf16, int grad_bf16,
                       int value_f32, hipStream_t stream) {
  const size_t lds = step_lds_bytes(p, value_f32);
  if (threads_for_block(p.block) == 64)
    return launch_dtypes<64, 16>(p, grid, lds, param_bf16, grad_bf16, value_f32, stream);
  return launch_dtypes<256, 16>(p, grid, lds, param_bf16, grad_bf16, value_f32, stream);
}

hipError_t launch_moments(const StepParams& p, int32_t tensor, int64_t first_block, int64_t grid,
                          float* mhat, float* vhat, int value_f32, hipStream_t stream) {
  const int nt = threads_for_block(p.block);
  StepParams q = p;
  q.stage_slots = 0;
  const size_t lds = step_lds_bytes(q, value_f32);
  if (nt == 64) {
    if (value_f32)
      hipLaunchKernelGGL((moments_kernel<64, true>), dim3((uint32_t)grid), dim3(64), lds, stream,
                         q, tensor, first_block, mhat, vhat);
    else
      hipLaunchKernelGGL((moments_kernel<64, false>), dim3((uint32_t)grid), dim3(64), lds, stream,
                         q, tensor, first_block, mhat, vhat);
  } else {
    if (value_f32)
      hipLaunchKernelGGL((moments_kernel<256, true>), dim3((uint32_t)grid), dim3(256), lds, stream,
                         q, tensor, first_block, mhat, vhat);
    else
      hipLaunchKernelGGL((moments_kernel<256, false>), dim3((uint32_t)grid), dim3(256), lds,
                         stream, q, tensor, first_block, mhat, vhat);
  }
  return hipGetLastError();
}

}  // namespace microadam
