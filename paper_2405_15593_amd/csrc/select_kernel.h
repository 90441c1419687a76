// The one-wave select kernel (steps 1-4 of a MicroAdam step for blocks of up
// to 4096 elements) and its launch templates.  Included by the translation
// units that instantiate it for one error-feedback format each.
#pragma once

#include "microadam_common.h"

namespace microadam {
namespace {

// Five waves per SIMD (96 registers; the kernel's 7.9 KB of LDS lets 20
// waves share a compute unit): measured 3% faster than four on the
// Llama-2-7B list (4.07 -> 3.95 ms), the few registers spilled included.
template <int EPL, bool LB, bool GBF16, bool VF32, int EFM, bool LQ = false>
__global__ void __launch_bounds__(kWave) __attribute__((amdgpu_waves_per_eu(5)))
select_kernel(StepParams p, int64_t first, int64_t count) {
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
  const int64_t gb = first + xcd_block(block_id(), count);

  // The block's EF codes and bucket pairs are addressed by gb alone, so their
  // loads go out before the tensor lookup that the gradient needs.
  const uint32_t nbk = (uint32_t)(p.block >> bl);
  const uint32_t ef_bytes = (EFM & kEf8) ? (uint32_t)p.block : (uint32_t)(p.block >> 1);
  const Rsrc re = make_rsrc(p.state + p.ef_plane + (uint64_t)gb * ef_bytes, ef_bytes);
  const Rsrc rs = make_rsrc(p.state + p.stats_plane + (uint64_t)gb * nbk * 8, nbk * 8);
  const bool wide = p.block == CAP;
  // 4096-element blocks of bf16 gradients with 4-bit codes load and store
  // the block as contiguous kilobytes and exchange it through LDS
  // (coalesced_exchange); the other shapes load each lane's run directly
  // (with 8-bit codes the exchange measured slower here: 5.95 vs 5.75 ms on
  // the Llama-2-7B list)
  constexpr bool kCoal = EPL == 64 && GBF16 && (EFM & kEf8) == 0 && !LQ;
  const bool coal = kCoal && wide;
  LaneIn<EPL, LB, GBF16, EFM> in;
  CoalescedIn cx;
  if constexpr (LQ) {
    lane_load_codes(in, re, eb, wide);
  } else if (coal) {
#pragma unroll
    for (int v = 0; v < (LB ? 1 : EPL / 8); ++v)
      in.st[v] = __builtin_amdgcn_raw_buffer_load_b64(rs, ((eb + 8 * v) >> bl) * 8, 0, kStream);
    coalesced_load_codes<EFM>(cx, re, lane);
  } else {
    lane_load_state(in, re, rs, eb, bl, wide);
  }
  const Block b = locate(p, gb);
  LqBuckets lqb = {};
  if constexpr (LQ) lqb = lq_buckets(p, b, eb, EPL, 0);
  const int s = b.s, kq = b.kq;
  const bool full = s == CAP;
  const Rsrc rg = make_rsrc((const uint8_t*)b.desc.grad + b.e0 * (GBF16 ? 2 : 4), vec_bytes<GBF16>(s));
  if (coal) coalesced_load_grad(cx, rg, lane);
  else lane_load_grad(in, rg, eb);
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
  const uint32_t edge_old = __builtin_amdgcn_raw_buffer_load_b32(rrec, edge_off, 0, kStream);
  if constexpr (kCoal) {
    if (coal) coalesced_exchange(cx, in, smem, lane);
  }

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
          __builtin_amdgcn_raw_buffer_store_b128(*(const u32x4*)(rowbuf + 4 * q), rrec, span_lo + 16 * q, 0,
                                                 kStream);
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
      // With finite keys exactly one lane has `mine`.  A NaN reaches no
      // threshold, so with fewer than k non-NaN keys none may have it: the
      // guard keeps the read defined, and the stores below stay in the row.
      const uint64_t mm = ballot(mine);
      i_last = mm ? __builtin_amdgcn_readlane(my_last, (int)__builtin_ctzll(mm)) : 0u;
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
            if (pos < (uint32_t)kq) E::store(rw, row0 + pos, E::make(eb + 8 * v + e, a[v][e]));
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
                                      EfStream{b.e0, b.j, (uint32_t)p.t, p.seed_lo, p.seed_hi},
                                      coal ? smem : nullptr);
  }
}

template <int EPL, bool LB, bool GB, bool VF, int EFM>
hipError_t launch_select_t(const StepParams& p, int64_t first, int64_t count, hipStream_t stream) {
  if (count <= 0) return hipSuccess;
  const size_t lds = select_lds_words() * 4;
  hipLaunchKernelGGL((select_kernel<EPL, LB, GB, VF, EFM>), dim3((uint32_t)count), dim3(kWave), lds, stream, p,
                     first, count);
  return hipGetLastError();
}

// Elements per lane of the select kernel: 16, 32 or 64.
inline int select_epl(int block) { return block <= 1024 ? 16 : block <= 2048 ? 32 : 64; }

template <int EPL, bool GB, bool VF, int EFM>
hipError_t launch_select_e(const StepParams& p, int64_t first, int64_t count, hipStream_t stream) {
  // whole buckets per lane (B_q >= EPL) or buckets of whole vectors
  if ((1 << p.bucket_log2) >= EPL) return launch_select_t<EPL, true, GB, VF, EFM>(p, first, count, stream);
  return launch_select_t<EPL, false, GB, VF, EFM>(p, first, count, stream);
}

// Blocks of up to 4096 elements in the error-feedback format EFM.
template <int EFM>
hipError_t launch_select_mode(const StepParams& p, int grad_bf16, int value_f32, int64_t first, int64_t count,
                              hipStream_t stream) {
  auto by_epl = [&](auto gb_tag, auto vf_tag) {
    constexpr bool GB = decltype(gb_tag)::value, VF = decltype(vf_tag)::value;
    switch (select_epl(p.block)) {
      case 16: return launch_select_e<16, GB, VF, EFM>(p, first, count, stream);
      case 32: return launch_select_e<32, GB, VF, EFM>(p, first, count, stream);
      default: return launch_select_e<64, GB, VF, EFM>(p, first, count, stream);
    }
  };
  using T = std::true_type;
  using F = std::false_type;
  if (grad_bf16) return value_f32 ? by_epl(T{}, T{}) : by_epl(T{}, F{});
  return value_f32 ? by_epl(F{}, T{}) : by_epl(F{}, F{});
}

}  // namespace
}  // namespace microadam
