// The update kernel for Top-K blocks above 4096 elements (one wave per run
// of 1024-element quarters of a block).
#include "microadam_common.h"

namespace microadam {
namespace {

// ================================================ update, blocks above 4096
// A wave takes kQuartersPerWave consecutive 1024-element quarters of a
// block, one after the other (lane l: the quarter's parameter vectors l and
// 64 + l, Vec16, so that each vector access of the wave is one contiguous
// kilobyte).
// The live rows' entries of quarter q are the segments the select kernel
// recorded in the record's table: row r holds them at positions
// [table(r, q), table(r, q + 1)).  For each quarter the wave loads every live
// row's segment at once (entry i of each segment's first 64 in lane i, and of
// the entries 64 .. 127 of up to kOverflow rows, while at most fast_rows()
// rows are live; else 64 entries of a row at a time), then adds them into two
// LDS accumulators, sum beta1^r V and sum beta2^r V^2 (Algorithm 2,
// AdamStats), the two sums of an element side by side in one 8-byte word:
// the entries of one add come from one row and have distinct indices, and
// the wave's LDS accesses execute in order, so every entry is added once,
// with no barrier.  Every lane then turns its 16 elements' sums into the
// update (an element without entries has sums 0 and keeps theta, less the
// decay) and applies it (Algorithm 1; Algorithm 4).  The loads of the next
// quarter (its table words, its segments and its parameters) go out before
// the current quarter is rebuilt, so their latency hides behind the rebuild.
// The decrement (eta*c1*s1) * rcp(eps + sqrt(c2*s2)) uses the hardware
// square root and reciprocal (each within 1 ulp), so it lies within a few
// binary32 ulps of the correctly rounded value.
constexpr int kQuartersPerWave = 4;
constexpr int kOverflow = 4;
constexpr int kPreRows = 8;  // rows of the next quarter loaded ahead
template <bool VF32>
constexpr int fast_rows() { return VF32 ? 12 : 24; }  // two quarters' entries stay in registers

// The accumulator: 8-byte (sum, sum) pairs in element order, and one sink
// pair (kQuarter) for entries outside the quarter, which the table rules
// out.
constexpr size_t update_large_lds_bytes() { return (size_t)(kQuarter + 2) * 8; }

// The loads of the next quarter that go out before the current one is
// rebuilt: its segments, its first kPreRows rows' entries and its parameters.
template <bool PBF16, bool VF32>
struct Prefetch {
  using ET = typename Entry<VF32>::T;
  uint32_t seg_lo, seg_n;  // lane r < n_live: row r's segment (first entry in the record, length)
  ET ld[kPreRows];
  u32x4 th[Vec16<PBF16>::NV];  // the lane's 16 parameters
};

template <bool PBF16, bool VF32, bool EXPORT>
__global__ void __launch_bounds__(kWave) update_large_kernel(StepParams p, int64_t first_block, int64_t count,
                                                             int32_t nw, float* mhat, float* vhat) {
  using E = Entry<VF32>;
  using ET = typename E::T;
  using PF = Prefetch<PBF16, VF32>;
  constexpr int FR = fast_rows<VF32>();
  extern __shared__ __align__(16) uint32_t smem[];
  float2* const z = (float2*)smem;  // [kQuarter + 1] (sum beta1^r V, sum beta2^r V^2)

  const int lane = thread_id();
  // the threshold kernel's list of unsettled blocks is used up: its count
  // starts the next step at 0 (the step's own update only, not a moment
  // export, which may run on another stream)
  if (!EXPORT && p.thr != nullptr && block_id() == 0 && lane == 0)
    __builtin_amdgcn_raw_buffer_store_b32(0u, make_rsrc(p.thr + thr_list_offset(p.total_blocks), 16), 0, 0, 0);
  const int64_t wg = xcd_block(block_id(), count * nw);
  const int32_t gb = (int32_t)(first_block + wg / nw);
  const int es = PBF16 ? 2 : 4;
  const Span g = span_of(p, gb, es);
  const int nqv = (g.s + kQuarter - 1) / kQuarter;  // quarters holding elements
  const int q_begin = (int)(wg % nw) * kQuartersPerWave;
  if (q_begin >= nqv) return;  // past the end of a ragged block
  const int q_end = q_begin + kQuartersPerWave < nqv ? q_begin + kQuartersPerWave : nqv;
  const int kq = g.kq, m = p.window, n_live = p.n_live;
  const int nq_blk = (p.block + kQuarter - 1) / kQuarter;  // table entries per row
  using V = Vec16<PBF16>;
  constexpr int EV = V::EV;
  // lane r < n_live: live row r (r = 0 is the oldest)
  const int my_slot = (p.new_slot + 1 + m - n_live + lane) % m;
  constexpr uint32_t EB = VF32 ? 8u : 4u;
  const Rsrc rrec = make_rsrc(p.state + p.win_plane + (uint64_t)gb * p.win_stride, (uint32_t)p.win_stride);
  const uint32_t table = (uint32_t)m * p.k_full * EB;
  const Rsrc rw = window_rsrc<VF32 ? 2 : 1>(p, gb, kq);
  const float lc1 = p.lr * p.c1;  // eta * (1 - beta1) / (1 - beta1^t)
  const float w1s = lane < kMaxWindow ? constant_ptr(p.wpow)[lane] : 0.0f;
  const float w2s = lane < kMaxWindow ? constant_ptr(p.wpow)[kMaxWindow + lane] : 0.0f;
  auto weight = [&](float ws, int r) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(ws), n_live - 1 - r));
  };
  auto quarter_size = [&](int q) { return g.s - q * kQuarter < kQuarter ? g.s - q * kQuarter : kQuarter; };
  auto param_rsrc = [&](int q) {
    return make_rsrc((const void*)(g.base + (uint64_t)q * kQuarter * es), vec_bytes<PBF16>(quarter_size(q)));
  };
  // entry `lane` + off of row r's segment, or (lanes past its end) a read
  // past the end of the record, which gives 0 and is not used: the adds
  // check the segment length, and no merge waits for the load.  (Default
  // cache policy: neighbouring quarters' segments share lines, which the nt
  // policy evicts early; measured on the 1.5e9 workload, nt here took the
  // kernel from 2.31 to 2.70 ms.)
  auto row_load = [&](uint32_t seg_lo, uint32_t seg_n, int r, uint32_t off) {
    const uint32_t n = __builtin_amdgcn_readlane(seg_n, r), at = __builtin_amdgcn_readlane(seg_lo, r);
    return E::load(rw, (uint32_t)lane + off < n ? at + off + (uint32_t)lane : E::kFar);
  };

  // the two table words of quarter q for the lane's row
  auto table_load = [&](int q, uint32_t& a0, uint32_t& a1) {
    a0 = 0u;
    a1 = 0u;
    if (lane < n_live) {
      a0 = __builtin_amdgcn_raw_buffer_load_b32(rrec, table + ((uint32_t)my_slot * nq_blk + q) * 4, 0, 0);
      a1 = q + 1 < nq_blk
               ? __builtin_amdgcn_raw_buffer_load_b32(rrec, table + ((uint32_t)my_slot * nq_blk + q + 1) * 4, 0, 0)
               : (uint32_t)kq;
    }
  };
  // quarter q's segments from its table words (clamped to the row, so that
  // any content gives a bounded read; lanes past the live rows hold empty
  // segments), then its prefetched loads issued
  auto open = [&](PF& F, int q, uint32_t a0, uint32_t a1) {
    const uint32_t b0 = a0 < (uint32_t)kq ? a0 : (uint32_t)kq, b1 = a1 < (uint32_t)kq ? a1 : (uint32_t)kq;
    F.seg_lo = lane < n_live ? (uint32_t)my_slot * kq + b0 : 0u;
    F.seg_n = lane < n_live && b1 > b0 ? b1 - b0 : 0u;
#pragma unroll
    for (int r = 0; r < kPreRows; ++r) F.ld[r] = row_load(F.seg_lo, F.seg_n, r, 0);
    if (!EXPORT) {
      const Rsrc rp = param_rsrc(q);
#pragma unroll
      for (int v = 0; v < V::NV; ++v) F.th[v] = V::load(rp, V::template first<kWave>(v, lane));
    }
  };

  // one entry's read-add-write of both sums (entries outside the quarter go
  // to the sink pair)
  auto add = [&](int lo, ET e, float w1, float w2) {
    const uint32_t zw = __builtin_elementwise_min(E::word(e) - (uint32_t)lo, (uint32_t)kQuarter);
    const float v = E::val(e);
    const float2 a = z[zw];
    z[zw] = make_float2(a.x + w1 * v, a.y + w2 * (v * v));
  };
  // quarter q rebuilt from its loads, then updated; `next` issues the next
  // quarter's prefetch once this quarter's own loads are out
  auto apply = [&](PF& F, int q, auto&& next) {
    const int lo = q * kQuarter, s = quarter_size(q);
    uint32_t longest = F.seg_n;
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
      const uint32_t o = __shfl_xor(longest, d, kWave);
      longest = longest > o ? longest : o;
    }
    longest = sgpr(longest);
    // rows with more than 64 entries in the quarter: their entries 64 .. 127
    // form a second chunk, added after every row's first chunk
    const uint64_t over = ballot(F.seg_n > (uint32_t)kWave);
    const int n_over = (int)popc(over);
    const bool fast = n_live <= FR && longest <= 2u * kWave && n_over <= kOverflow;
    // the rest of the rows and the second chunks
    ET ld[FR - kPreRows], lx[kOverflow];
    int xr[kOverflow];
#pragma unroll
    for (int r = kPreRows; r < FR; ++r) ld[r - kPreRows] = row_load(F.seg_lo, F.seg_n, r, 0);
    uint64_t om = over;
#pragma unroll
    for (int j = 0; j < kOverflow; ++j) {
      const int r = om ? (int)__builtin_ctzll(om) : 0;
      om &= om - 1;
      xr[j] = r;
      lx[j] = row_load(F.seg_lo, j < n_over ? F.seg_n : 0u, r, kWave);
    }
    const uint32_t seg_lo = F.seg_lo, seg_n = F.seg_n;
    ET pre[kPreRows];
#pragma unroll
    for (int r = 0; r < kPreRows; ++r) pre[r] = F.ld[r];
    u32x4 th[V::NV];
#pragma unroll
    for (int v = 0; v < V::NV; ++v) th[v] = F.th[v];
    next();
    {
      const float4 zero = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
      for (int w = 0; w < 8; ++w) *(float4*)(z + w * 2 * kWave + lane * 2) = zero;
    }
    wave_sync();  // the cleared accumulators before any entry is added
    if (fast) {
      // (one row's arithmetic at a time: the adds are a chain through LDS,
      // and arithmetic hoisted ahead of it only holds registers)
#pragma unroll
      for (int r = 0; r < FR; ++r) {
        if ((uint32_t)lane < __builtin_amdgcn_readlane(seg_n, r))
          add(lo, r < kPreRows ? pre[r] : ld[r - kPreRows], weight(w1s, r), weight(w2s, r));
        __builtin_amdgcn_sched_barrier(0);
      }
#pragma unroll
      for (int j = 0; j < kOverflow; ++j) {
        if (j < n_over && (uint32_t)lane + kWave < __builtin_amdgcn_readlane(seg_n, xr[j]))
          add(lo, lx[j], weight(w1s, xr[j]), weight(w2s, xr[j]));
        __builtin_amdgcn_sched_barrier(0);
      }
    } else {
      for (int r = 0; r < n_live; ++r) {
        const uint32_t n = __builtin_amdgcn_readlane(seg_n, r), at = __builtin_amdgcn_readlane(seg_lo, r);
        const float w1 = weight(w1s, r), w2 = weight(w2s, r);
        for (uint32_t x = (uint32_t)lane; x < n; x += kWave) add(lo, E::load(rw, at + x), w1, w2);
      }
    }
    wave_sync();
    if ((int)V::template first<kWave>(0, lane) >= s) return;
    const bool full = s == kQuarter;
#pragma unroll
    for (int v = 0; v < V::NV; ++v) {
      const uint32_t e0 = V::template first<kWave>(v, lane);
      float s1[EV], s2[EV];
#pragma unroll
      for (int w = 0; w < EV / 2; ++w) {
        const float4 u = *(const float4*)(z + e0 + 2 * w);  // elements e0 + 2w, + 1
        s1[2 * w] = u.x; s2[2 * w] = u.y; s1[2 * w + 1] = u.z; s2[2 * w + 1] = u.w;
      }
      if (EXPORT) {
#pragma unroll
        for (int e = 0; e < EV; ++e)
          if ((int)e0 + e < s) {
            mhat[g.e0 + lo + e0 + e] = p.c1 * s1[e];
            vhat[g.e0 + lo + e0 + e] = p.c2 * s2[e];
          }
        continue;
      }
      float thf[EV], out[EV];
      V::unpack(th[v], thf);
#pragma unroll
      for (int e = 0; e < EV; ++e) {
        // an element without entries has s1 = s2 = 0, so its decrement is
        // 0 * rcp(eps) = 0: no separate test
        const float den = p.eps + __builtin_amdgcn_sqrtf(p.c2 * s2[e]);
        const float d = (lc1 * s1[e]) * __builtin_amdgcn_rcpf(den);
        const float base = thf[e] * p.decay;  // exact when the factor is 1
        out[e] = base - d;
      }
      V::store(param_rsrc(q), e0, s, full, out);
    }
  };

  // quarter q + 1's prefetch goes out before quarter q is rebuilt, and
  // quarter q + 2's table words with it
  PF A, B;
  uint32_t t0, t1;
  table_load(q_begin, t0, t1);
  open(A, q_begin, t0, t1);
  if (q_begin + 1 < q_end) table_load(q_begin + 1, t0, t1);
  auto step = [&](PF& cur, PF& nxt, int q) {
    apply(cur, q, [&]() {
      if (q + 1 < q_end) {
        open(nxt, q + 1, t0, t1);
        if (q + 2 < q_end) table_load(q + 2, t0, t1);
      }
    });
  };
  for (int q = q_begin; q < q_end; q += 2) {
    step(A, B, q);
    if (q + 1 < q_end) step(B, A, q + 1);
  }
}

// Waves of kQuartersPerWave quarters over each block of [first, first + count).
template <bool PB, bool VF, bool EXPORT>
hipError_t launch_update_large(const StepParams& p, int64_t first, int64_t count, float* mh, float* vh,
                               hipStream_t stream) {
  if (count <= 0) return hipSuccess;
  const int32_t nq = (p.block + kQuarter - 1) / kQuarter;
  const int32_t nw = (nq + kQuartersPerWave - 1) / kQuartersPerWave;
  hipLaunchKernelGGL((update_large_kernel<PB, VF, EXPORT>), dim3((uint32_t)(count * nw)), dim3(kWave),
                     update_large_lds_bytes(), stream, p, first, count, nw, mh, vh);
  return hipGetLastError();
}

}  // namespace

size_t update_large_lds() { return update_large_lds_bytes(); }

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
