// Steps with quantization buckets spanning Top-K blocks: the select kernel's
// partials form, the bucket reduction and the second quantization pass.
#include "select_kernel.h"
#include "select_large_kernel.h"

namespace microadam {
namespace {

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
// 4096-element sub-block of a block (the whole block up to 4096 elements),
// 64 elements per lane.  Above 4096 the sub-block's entries of the new row
// are those of its four 1024-element quarters, found through the record's
// segment table.
template <bool GBF16, bool VF32, int EFM>
__global__ void __launch_bounds__(kWave) __attribute__((amdgpu_waves_per_eu(4)))
requant_kernel(StepParams p, int64_t first, int64_t count, int32_t nsub) {
  constexpr int EPL = 64, NV = EPL / 8, CAP = kWave * EPL;
  constexpr int CW = (EFM & kEf8) ? 2 : 1;
  using E = Entry<VF32>;
  __shared__ uint32_t kept[CAP / 32];  // bit i: element off + i is in the new row

  const int lane = thread_id();
  const int64_t w = xcd_block(block_id(), count * nsub);
  const int64_t gb = first + w / nsub;
  const uint32_t off = (uint32_t)(w % nsub) * CAP;  // the sub-block's first element
  const uint32_t eb = off + (uint32_t)lane * EPL;   // the lane's first element in the block
  const uint32_t ef_bytes = (EFM & kEf8) ? (uint32_t)p.block : (uint32_t)(p.block >> 1);
  const Rsrc re = make_rsrc(p.state + p.ef_plane + (uint64_t)gb * ef_bytes, ef_bytes);
  // 16-byte code accesses when no lane's codes straddle the end of the block's
  const bool wide = p.block % CAP == 0;
  LaneIn<EPL, true, GBF16, EFM> in;
  lane_load_codes(in, re, eb, wide);
  const Block b = locate(p, gb);
  const int s = b.s, kq = b.kq;
  if ((int)off >= s) return;  // a sub-block past the end of a ragged block
  const bool full = s - (int)off >= CAP;
  const Rsrc rg = make_rsrc((const uint8_t*)b.desc.grad + b.e0 * (GBF16 ? 2 : 4), vec_bytes<GBF16>(s));
  lane_load_grad(in, rg, eb);
  const LqBuckets old_b = lq_buckets(p, b, eb, EPL, 0), new_b = lq_buckets(p, b, eb, EPL, 1);

  kept[lane] = 0u;
  kept[lane + kWave] = 0u;
  wave_sync();
  const Rsrc rw = window_rsrc<VF32 ? 2 : 1>(p, gb, kq);
  const uint32_t row0 = (uint32_t)p.new_slot * kq;
  // the row's entries of this sub-block: [j0, j1)
  uint32_t j0 = 0, j1 = (uint32_t)kq;
  if (p.block > CAP) {
    constexpr uint32_t EB = VF32 ? 8u : 4u;
    const int nq = (p.block + kQuarter - 1) / kQuarter;
    const int q0 = (int)(off / kQuarter), q1 = q0 + CAP / kQuarter;
    const Rsrc rrec = make_rsrc(p.state + p.win_plane + (uint64_t)gb * p.win_stride, (uint32_t)p.win_stride);
    const uint32_t table = (uint32_t)p.window * p.k_full * EB + (uint32_t)p.new_slot * nq * 4;
    const uint32_t a0 = __builtin_amdgcn_raw_buffer_load_b32(rrec, table + (uint32_t)q0 * 4, 0, 0);
    const uint32_t a1 = q1 < nq ? __builtin_amdgcn_raw_buffer_load_b32(rrec, table + (uint32_t)q1 * 4, 0, 0)
                                : (uint32_t)kq;
    j0 = sgpr(a0 < (uint32_t)kq ? a0 : (uint32_t)kq);  // clamped: any content gives a bounded read
    j1 = sgpr(a1 < (uint32_t)kq ? a1 : (uint32_t)kq);
  }
  for (uint32_t j = j0 + (uint32_t)lane; j < j1; j += kWave) {
    const uint32_t i = E::idx(E::load(rw, row0 + j)) - off;
    if (i < (uint32_t)CAP) atomicOr(&kept[i >> 5], 1u << (i & 31));
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

template <bool GB, bool VF, int EF8>
hipError_t launch_select_partials_t(const StepParams& p, hipStream_t stream) {
  if (p.block > kSubBlock) return launch_select_large<GB, VF, EF8, true>(p, 0, p.total_blocks, stream);
  const size_t lds = select_lds_words() * 4;
  hipLaunchKernelGGL((select_kernel<64, true, GB, VF, EF8, true>), dim3((uint32_t)p.total_blocks), dim3(kWave), lds,
                     stream, p, (int64_t)0, p.total_blocks);
  return hipGetLastError();
}

template <bool GB, bool VF>
hipError_t launch_select_partials_d(const StepParams& p, hipStream_t stream) {
  return (p.ef_mode & kEf8) ? launch_select_partials_t<GB, VF, kEf8>(p, stream)
                            : launch_select_partials_t<GB, VF, 0>(p, stream);
}

template <bool GB, bool VF, int EFM>
hipError_t launch_requant_t(const StepParams& p, hipStream_t stream) {
  const int32_t nsub = (p.block + kSubBlock - 1) / kSubBlock;
  hipLaunchKernelGGL((requant_kernel<GB, VF, EFM>), dim3((uint32_t)(p.total_blocks * nsub)), dim3(kWave), 0, stream,
                     p, (int64_t)0, p.total_blocks, nsub);
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
