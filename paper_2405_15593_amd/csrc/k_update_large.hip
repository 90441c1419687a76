// The update kernel for Top-K blocks above 4096 elements (one workgroup per
// 4096-element sub-block).
#include "microadam_common.h"

namespace microadam {
namespace {

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
__global__ void __launch_bounds__(256) update_large_kernel(StepParams p, int64_t first_block, int64_t count, int32_t nsub,
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
  const int64_t wg = xcd_block(block_id(), count * nsub);
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
      // (segment starts are clamped to the row, so that any table content
      // gives a bounded read)
      const uint32_t b0 = a0 < (uint32_t)kq ? a0 : (uint32_t)kq, b1 = a1 < (uint32_t)kq ? a1 : (uint32_t)kq;
      start = (uint32_t)slot * kq + b0;  // entry number in the record
      n = b1 > b0 ? b1 - b0 : 0u;
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
      const float den = p.eps + __builtin_sqrtf(vh);  // correctly rounded
      // an element without entries is left to the decay alone
      const bool none = (s1[8 * v + e] == 0.0f) & (s2[8 * v + e] == 0.0f);
      const float d = none ? 0.0f : p.lr * (mh / den);
      const float base = p.decay_is_one ? thf[e] : thf[e] * p.decay;
      out[e] = base - d;
    }
    store8<PBF16>(rp, eb + 8 * v, s, full, out);
  }
}

// One workgroup per 4096-element sub-block of each block of [first, first + count).
template <bool PB, bool VF, bool EXPORT>
hipError_t launch_update_large(const StepParams& p, int64_t first, int64_t count, float* mh, float* vh,
                               hipStream_t stream) {
  if (count <= 0) return hipSuccess;
  const int32_t nsub = (p.block + kSubBlock - 1) / kSubBlock;
  hipLaunchKernelGGL((update_large_kernel<PB, VF, EXPORT>), dim3((uint32_t)(count * nsub)), dim3(256),
                     update_large_lds_bytes<VF>(), stream, p, first, count, nsub, mh, vh);
  return hipGetLastError();
}

}  // namespace

size_t update_large_lds() { return update_large_lds_bytes<true>(); }

hipError_t launch_update_large_blocks(const StepParams& p, int param_bf16, int value_f32, int64_t first,
                                      int64_t count, hipStream_t stream) {
  if (param_bf16)
    return value_f32 ? launch_update_large<true, true, false>(p, first, count, nullptr, nullptr, stream)
                     : launch_update_large<true, false, false>(p, first, count, nullptr, nullptr, stream);
  return value_f32 ? launch_update_large<false, true, false>(p, first, count, nullptr, nullptr, stream)
                   : launch_update_large<false, false, false>(p, first, count, nullptr, nullptr, stream);
}

hipError_t launch_moments_large_blocks(const StepParams& p, int64_t first_block, int64_t num_blocks, float* mhat,
                                       float* vhat, int value_f32, hipStream_t stream) {
  return value_f32 ? launch_update_large<false, true, true>(p, first_block, num_blocks, mhat, vhat, stream)
                   : launch_update_large<false, false, true>(p, first_block, num_blocks, mhat, vhat, stream);
}

}  // namespace microadam
