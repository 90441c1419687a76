// The multi-wave select kernel for Top-K blocks above 4096 elements and its
// launch templates.  Included by the translation units that instantiate it
// for one error-feedback format each.
#pragma once

#include "microadam_common.h"
#include "select_split_kernel.h"

namespace microadam {
namespace {

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
// and for each 1024-element quarter of the block the position in the row of
// its first entry goes to the record's segment table, behind the m rows,
// where the update finds the entries of one quarter.
constexpr int kCandPerThread = 8;
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

// LQ: buckets spanning blocks -- the decode takes each lane's two buckets
// from the bucket table, and the block ends with its partials (the (min, max)
// of the residual in its first bucket and in the next one, over all waves)
// instead of the codes, which a second pass quantizes.
template <int NW, bool LB, bool GBF16, bool VF32, int EFM, bool LQ>
__device__ __forceinline__ void select_large_block(const StepParams& p, int64_t gb) {
  constexpr int EPL = 64, NV = 8, NT = NW * kWave, CAP = NT * EPL, R = kCandPerThread, NC = NT * R;
  constexpr int SPT = kSamples / NT, SPL = kSamples / kWave;  // samples per thread; per lane
  constexpr int DPW = 16 / NW;                                  // sample digits per wave
  static_assert(SPT >= 1 && SPT <= NV, "one to eight samples per thread");
  static_assert(!LQ || (LB && (EFM & kEfRandom) == 0), "buckets spanning blocks: the decode has no random draws");
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

  // ---------------------------------------------- 1. a = g + Q^-1(e)
  float a[NV][8];
  const int rem = s - (int)eb;
  if constexpr (LQ) lane_decode_lq(in, lqb, a, rem, full);
  else lane_decode(in, a, rem, full);

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
      for (int r = 0; r < R; ++r) m_l += ((y[r] >= t1) & (y[r] < U)) ? 1u : 0u;
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
    // (misc[0] holds 0 unless a thread below writes it: with finite keys
    // exactly one does; with NaNs, which reach no bound, possibly none)
    if (tid == 0) misc[0] = 0u;
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
    // the new row in element order, and the segment table entries of the
    // block's 1024-element quarters: the row position of each quarter's first
    // entry, written by the thread holding the quarter's first 64 elements
    uint32_t kept_all;
    uint32_t pos = wg_scan(sel_l, 1, kept_all);
    constexpr uint32_t EB = VF32 ? 8u : 4u;
    const int nq = (p.block + kQuarter - 1) / kQuarter;
    const Rsrc rrec = make_rsrc(p.state + p.win_plane + (uint64_t)gb * p.win_stride, (uint32_t)p.win_stride);
    if ((tid & (kQuarter / EPL - 1)) == 0 && tid / (kQuarter / EPL) < nq)
      __builtin_amdgcn_raw_buffer_store_b32(
          pos < (uint32_t)kq ? pos : (uint32_t)kq, rrec,
          (uint32_t)p.window * p.k_full * EB + ((uint32_t)p.new_slot * nq + tid / (kQuarter / EPL)) * 4, 0, 0);
    // the row goes through LDS (the gathered keys are no longer needed)
    // when it fits, and leaves in whole-wave stores of consecutive words;
    // else each entry is stored where it is found
    constexpr uint32_t EW = VF32 ? 2u : 1u;
    const bool staged = (uint32_t)kq * EW <= (uint32_t)NC;
    const Rsrc rw = window_rsrc<VF32 ? 2 : 1>(p, gb, kq);
    const uint32_t row0 = (uint32_t)p.new_slot * kq;
    if (sel_l) {
      const float tf = opaque_f(__uint_as_float(T));
      const int last_here = notie ? CAP : (int)i_last - (int)eb;
#pragma unroll
      for (int v = 0; v < NV; ++v) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float ab = __builtin_fabsf(a[v][e]);
          if ((ab > tf) | ((ab == tf) & (8 * v + e <= last_here))) {
            if (pos < (uint32_t)kq) {  // within the row
              const typename E::T x = E::make(eb + 8 * v + e, a[v][e]);
              if (staged) {
                if constexpr (VF32) *(u32x2*)(region + 2 * pos) = x;
                else region[pos] = x;
              } else {
                E::store(rw, row0 + pos, x);
              }
            }
            ++pos;
          }
        }
        __builtin_amdgcn_sched_barrier(0);  // one vector's stores at a time
      }
    }
    if (staged) {
      lds_sync();
      for (uint32_t w = (uint32_t)tid; w < (uint32_t)kq * EW; w += NT)
        __builtin_amdgcn_raw_buffer_store_b32(region[w], rw, (row0 * EW + w) * 4, 0, 0);
    }
  }

  // ---------------------------------------------- 4. e = Q(a with a[I] = 0)
  if constexpr (LQ) {
    lane_zero_kept<EPL>(a, T, notie, i_last, eb);
    // the waves' partials combined in LDS (dig is free since the search)
    float x[4];
    wave_partials<EPL>(a, p, b, eb, rem, x);
    if (lane == 0) {
#pragma unroll
      for (int c = 0; c < 4; ++c) dig[4 * wave + c] = __float_as_uint(x[c]);
    }
    lds_sync();
    if (tid == 0) {
#pragma unroll
      for (int w = 1; w < NW; ++w) {
        x[0] = __builtin_fminf(x[0], __uint_as_float(dig[4 * w]));
        x[1] = __builtin_fmaxf(x[1], __uint_as_float(dig[4 * w + 1]));
        x[2] = __builtin_fminf(x[2], __uint_as_float(dig[4 * w + 2]));
        x[3] = __builtin_fmaxf(x[3], __uint_as_float(dig[4 * w + 3]));
      }
      store_partials(p, gb, x);
    }
  } else {
    lane_quantize_store<EPL, LB, EFM>(a, T, notie, i_last, eb, s, rem, full, bl, wide, re, rs,
                                      EfStream{b.e0, b.j, (uint32_t)p.t, p.seed_lo, p.seed_hi});
  }
}

// One workgroup per block of [first, first + count).
template <int NW, bool LB, bool GBF16, bool VF32, int EFM, bool LQ = false>
__global__ void __launch_bounds__(NW * kWave) select_large_kernel(StepParams p, int64_t first, int64_t count) {
  select_large_block<NW, LB, GBF16, VF32, EFM, LQ>(p, first + xcd_block(block_id(), count));
}

// After the threshold and apply kernels: the blocks they could not settle,
// from their list, each workgroup taking every gridDim-th one.
template <int NW, bool LB, bool GBF16, bool VF32, int EFM>
__global__ void __launch_bounds__(NW * kWave) select_large_list_kernel(StepParams p) {
  const uint32_t* const list = (const uint32_t*)(p.thr + thr_list_offset(p.total_blocks));
  // (the count and the entries are bounded by the number of blocks, so that
  // any content of the list gives in-bounds work)
  const uint32_t n0 = sgpr(list[0]);
  const uint32_t n = n0 < (uint64_t)p.total_blocks ? n0 : (uint32_t)p.total_blocks;
  for (uint32_t i = (uint32_t)block_id(); i < n; i += gridDim.x) {
    const uint32_t gb = sgpr(list[4 + i]);
    if (gb < (uint64_t)p.total_blocks) select_large_block<NW, LB, GBF16, VF32, EFM, false>(p, (int64_t)gb);
    lds_sync();  // the block's last LDS reads before the next block's first writes
  }
}

// Waves of the large-block select kernel: 4096 elements each, 2 to 16.
inline int large_waves(int block) {
  const int w = (block + kSubBlock - 1) / kSubBlock;
  return w <= 2 ? 2 : w <= 4 ? 4 : w <= 8 ? 8 : 16;
}

template <int NW, bool GB, bool VF, int EFM, bool LQ = false>
hipError_t launch_select_large_t(const StepParams& p, int64_t first, int64_t count, hipStream_t stream) {
  if (count <= 0) return hipSuccess;
  const size_t lds = LargeLds<NW>::words() * 4;
  if constexpr (LQ)
    hipLaunchKernelGGL((select_large_kernel<NW, true, GB, VF, EFM, true>), dim3((uint32_t)count), dim3(NW * kWave),
                       lds, stream, p, first, count);
  else if ((1 << p.bucket_log2) >= 64)
    hipLaunchKernelGGL((select_large_kernel<NW, true, GB, VF, EFM>), dim3((uint32_t)count), dim3(NW * kWave), lds, stream,
                       p, first, count);
  else
    hipLaunchKernelGGL((select_large_kernel<NW, false, GB, VF, EFM>), dim3((uint32_t)count), dim3(NW * kWave), lds,
                       stream, p, first, count);
  return hipGetLastError();
}

template <bool GB, bool VF, int EFM, bool LQ = false>
hipError_t launch_select_large(const StepParams& p, int64_t first, int64_t count, hipStream_t stream) {
  switch (large_waves(p.block)) {
    case 2: return launch_select_large_t<2, GB, VF, EFM, LQ>(p, first, count, stream);
    case 4: return launch_select_large_t<4, GB, VF, EFM, LQ>(p, first, count, stream);
    case 8: return launch_select_large_t<8, GB, VF, EFM, LQ>(p, first, count, stream);
    default: return launch_select_large_t<16, GB, VF, EFM, LQ>(p, first, count, stream);
  }
}

// The multi-wave select over the list of blocks the threshold kernel could
// not settle: at most one workgroup per compute unit's worth of them, each
// taking every gridDim-th entry (an empty list costs one short launch).
template <int NW, bool GB, bool VF, int EFM>
hipError_t launch_select_large_list_t(const StepParams& p, hipStream_t stream) {
  const size_t lds = LargeLds<NW>::words() * 4;
  const uint32_t grid = (uint32_t)(p.total_blocks < 256 ? p.total_blocks : 256);
  if ((1 << p.bucket_log2) >= 64)
    hipLaunchKernelGGL((select_large_list_kernel<NW, true, GB, VF, EFM>), dim3(grid), dim3(NW * kWave), lds, stream, p);
  else
    hipLaunchKernelGGL((select_large_list_kernel<NW, false, GB, VF, EFM>), dim3(grid), dim3(NW * kWave), lds, stream, p);
  return hipGetLastError();
}

// Blocks above 4096 elements in the error-feedback format EFM: with
// threshold records (p.thr) and the whole step in one launch range, the
// threshold and apply kernels, then the multi-wave select for the blocks
// they left (their list); else the multi-wave select for every block.
template <bool GB, bool VF, int EFM>
hipError_t launch_select_large_all(const StepParams& p, int64_t first, int64_t count, hipStream_t stream) {
  if (p.thr == nullptr || first != 0 || count != p.total_blocks)
    return launch_select_large<GB, VF, EFM>(p, first, count, stream);
  const hipError_t e = launch_select_split<GB, VF, EFM>(p, first, count, stream);
  if (e != hipSuccess) return e;
  switch (large_waves(p.block)) {
    case 2: return launch_select_large_list_t<2, GB, VF, EFM>(p, stream);
    case 4: return launch_select_large_list_t<4, GB, VF, EFM>(p, stream);
    case 8: return launch_select_large_list_t<8, GB, VF, EFM>(p, stream);
    default: return launch_select_large_list_t<16, GB, VF, EFM>(p, stream);
  }
}

template <int EFM>
hipError_t launch_select_large_mode(const StepParams& p, int grad_bf16, int value_f32, int64_t first, int64_t count,
                                    hipStream_t stream) {
  if (grad_bf16)
    return value_f32 ? launch_select_large_all<true, true, EFM>(p, first, count, stream)
                     : launch_select_large_all<true, false, EFM>(p, first, count, stream);
  return value_f32 ? launch_select_large_all<false, true, EFM>(p, first, count, stream)
                   : launch_select_large_all<false, false, EFM>(p, first, count, stream);
}

}  // namespace
}  // namespace microadam
