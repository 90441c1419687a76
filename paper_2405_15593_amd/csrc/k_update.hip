// The update kernel for Top-K blocks of up to 4096 elements: the moment
// rebuild from the window and the parameter update, one workgroup per block.
#include "microadam_common.h"

namespace microadam {
namespace {

// ============================================================ update
// The accumulators hold, per element of the block, sum beta1^r V and sum
// beta2^r V^2 (z1 and z2; or z1 alone, one after the other), then z1 the
// parameter decrement.  A thread's 16 elements are its parameter vectors
// (Vec16: vector v of thread t holds the EV elements from v*EV*NT + t*EV),
// read as four groups of four: group g of thread t is the 16-byte word at
// (g*NT + t)*4, so a wave's 16-byte accesses fall on consecutive addresses.
// Element i = v*EV*NT + t*EV + e lies in group v*EV/4 + e/4, at word e mod 4
// (for binary32 parameters that is word i itself).  Word CAP of each array
// is a sink for lanes without an entry, which keeps the sparse updates free
// of branches.
template <int NT, bool PBF16>
__device__ __forceinline__ uint32_t zpos(uint32_t i) {
  constexpr uint32_t EV = Vec16<PBF16>::EV, G = EV / 4;
  const uint32_t v = i / (EV * NT), t = (i / EV) & (NT - 1), e = i & (EV - 1);
  return ((v * G + e / 4) * NT + t) * 4 + (e & 3);
}

// LDS: the accumulators (two, or one with ONE).
template <int NT, bool VF, int KC, bool ONE>
constexpr size_t update_lds_bytes() {
  return (size_t)(ONE ? 1 : 2) * (NT * kLaneElems + 16) * 4;
}

// One workgroup per block.  One wave (rotating with the block) rebuilds the
// moments of the block's window entries, oldest row first, and turns them
// into parameter decrements; then every thread updates its own elements.
//
// The leader loads the window entries straight into registers, KC chunks of
// 64 in the order it adds them: lane l of chunk c holds position 64*c + l,
// where chunk c is part c mod R of the live row c / R (oldest row first,
// R = ceil(k_q/64) parts of 64 entries); positions without an entry add into
// the sink word CAP.  A block whose live rows need more than KC chunks is
// read by the leader row by row from the window record.  The other waves
// load only their parameters.
//
// ONE = true: one accumulator; the leader makes two passes over its
// entries (first moments, read back and cleared, then second moments), which
// halves the LDS of a workgroup so that eight fit on a compute unit.  The
// host launches it only where every block's live rows fit in KC chunks.
// ONE = false: two accumulators, any block.  EXPORT = true writes dense m-hat
// and v-hat instead of updating theta.
// Waves per SIMD that the LDS of an update workgroup allows (160 KB per
// compute unit, four SIMDs); telling the compiler lets it spend registers
// up to that occupancy on keeping LDS reads in flight.  A leader holding 16
// chunks needs more than the 64 registers of eight waves per SIMD, so those
// kernels ask for seven.
template <int NT, bool VF, int KC, bool ONE>
constexpr int update_waves_per_eu() {
  const int per_cu = (int)(163840 / update_lds_bytes<NT, VF, KC, ONE>());
  const int w = per_cu * (NT / kWave) / 4;
  const int cap = KC >= 16 ? 7 : 8;
  return w < 1 ? 1 : w > cap ? cap : w;
}

template <int NT, bool PBF16, bool VF32, bool EXPORT, int KC, bool ONE>
__global__ void __launch_bounds__(NT) __attribute__((amdgpu_waves_per_eu(update_waves_per_eu<NT, VF32, KC, ONE>())))
update_kernel(StepParams p, int64_t first_block, int64_t count, float* mhat, float* vhat) {
  static_assert(!ONE || !EXPORT, "one accumulator: parameter update only");
  constexpr int NW = NT / kWave;
  constexpr int CAP = NT * kLaneElems;
  constexpr int kChunks = KC;                             // 64-entry chunks the leader holds
  using E = Entry<VF32>;
  using ET = typename E::T;
  extern __shared__ __align__(16) uint32_t smem[];
  float* const z1 = (float*)smem;
  float* const z2 = z1 + CAP + 16;                        // not allocated with ONE

  const int tid = thread_id(), lane = tid & (kWave - 1), wave = (int)sgpr(tid / kWave);
  const int m = p.window, n_live = p.n_live;
  // oldest live row first: the row written at step s is slot (s-1) mod m
  const int slot0 = (p.new_slot + 1 + m - n_live) % m;

  const Span u = span_of(p, (int32_t)(first_block + xcd_block(block_id(), count)), PBF16 ? 2 : 4);
  const int s = u.s, kq = u.kq;
  const int leader = u.gb & (NW - 1);
  const int R = (kq + kWave - 1) / kWave;
  const bool held = n_live * R <= kChunks;  // the leader holds every live chunk in registers

  // loads: the leader's window positions, KC chunks of 64 (positions without
  // an entry read entry 0 and are not used), then every thread's parameters.
  // Chunk c is part `col` of live row `row` (uniform counters), at record
  // entry slot*k_q + 64*col + lane.
  const bool lead = wave == leader;
  const Rsrc rw = window_rsrc<VF32 ? 2 : 1>(p, u.gb, kq);
  ET w[kChunks];
  bool has[kChunks];  // the position holds an entry
  int rr[kChunks];    // the chunk's row age: 0 for the newest row
  if (lead && held) {
    int row = 0, col = 0, slot = slot0;
#pragma unroll
    for (int c = 0; c < kChunks; ++c) {
      const int jj = col * kWave + lane;
      has[c] = row < n_live && jj < kq;
      rr[c] = (n_live - 1 - row) & (kMaxWindow - 1);
      w[c] = E::template load<kStream>(rw, has[c] ? (uint32_t)(slot * kq + jj) : 0u);
      if (++col == R) {
        col = 0;
        ++row;
        if (++slot == m) slot = 0;
      }
    }
  }
  using V = Vec16<PBF16>;
  constexpr int EV = V::EV;
  const Rsrc rp = make_rsrc((const void*)u.base, vec_bytes<PBF16>(s));
  u32x4 th[V::NV];
  if (!EXPORT) {
#pragma unroll
    for (int v = 0; v < V::NV; ++v) th[v] = V::load(rp, V::template first<NT>(v, tid));
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
  lds_sync();

  if (lead) {
    auto step_of = [&](float s1, float s2) {
      const float mh = p.c1 * s1;
      const float vh = p.c2 * s2;
      // correctly rounded square root and division
      const float den = p.eps + __builtin_sqrtf(vh);
      return p.lr * (mh / den);
    };
    if (held) {
      // chunks past the live rows hold only sink words
      uint32_t zp[kChunks];
      float val[kChunks];
#pragma unroll
      for (int c = 0; c < kChunks; ++c) {
        const uint32_t idx = E::idx(w[c]);
        zp[c] = has[c] && idx < (uint32_t)s ? zpos<NT, PBF16>(idx) : (uint32_t)CAP;
        val[c] = E::val(w[c]);
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
          const uint32_t zp = i < (uint32_t)s ? zpos<NT, PBF16>(i) : (uint32_t)CAP;
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
              const uint32_t zp = zpos<NT, PBF16>(i);
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
        const uint32_t i = V::template first<NT>(q / (EV / 4), tid) + (q % (EV / 4)) * 4 + r;
        if ((int)i < s) {
          mhat[u.e0 + i] = p.c1 * a1[r];
          vhat[u.e0 + i] = p.c2 * a2[r];
        }
      }
    }
    return;
  }

  // ------------------------------------------------ 6. parameter update
  // (theta times the decay factor, skipped by a uniform branch when the
  // factor is 1)
  const bool full = s == NT * kLaneElems;
  auto apply = [&](auto one_tag) {
    constexpr bool ONE_DECAY = decltype(one_tag)::value;
#pragma unroll
    for (int v = 0; v < V::NV; ++v) {
      const uint32_t e0 = V::template first<NT>(v, tid);  // vectors past s store nothing
      float upd[EV], thf[EV], out[EV];
#pragma unroll
      for (int q = 0; q < EV / 4; ++q) {
        const float4 x = *(const float4*)(z1 + ((v * (EV / 4) + q) * NT + tid) * 4);
        upd[4 * q] = x.x;
        upd[4 * q + 1] = x.y;
        upd[4 * q + 2] = x.z;
        upd[4 * q + 3] = x.w;
      }
      V::unpack(th[v], thf);
#pragma unroll
      for (int e = 0; e < EV; ++e) out[e] = (ONE_DECAY ? thf[e] : thf[e] * p.decay) - upd[e];
      V::store(rp, e0, s, full, out);
    }
  };
  if (p.decay_is_one)
    apply(BoolTag<true>{});
  else
    apply(BoolTag<false>{});
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
                     first, count, (float*)nullptr, (float*)nullptr);
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
                     p, first_block, blocks, mh, vh);
  return hipGetLastError();
}

}  // namespace

size_t update_lds_max(int nt) {
  return nt == 64 ? update_lds_bytes<64, true, 16, false>() : update_lds_bytes<256, true, 16, false>();
}

hipError_t launch_update_blocks(const StepParams& p, int param_bf16, int value_f32, int64_t first, int64_t count,
                                hipStream_t stream) {
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

hipError_t launch_moments_blocks(const StepParams& p, int64_t first_block, int64_t num_blocks, float* mhat,
                                 float* vhat, int value_f32, hipStream_t stream) {
  if (threads_for_block(p.block) == 64)
    return value_f32 ? launch_export<64, true>(p, first_block, num_blocks, mhat, vhat, stream)
                     : launch_export<64, false>(p, first_block, num_blocks, mhat, vhat, stream);
  return value_f32 ? launch_export<256, true>(p, first_block, num_blocks, mhat, vhat, stream)
                   : launch_export<256, false>(p, first_block, num_blocks, mhat, vhat, stream);
}

}  // namespace microadam
