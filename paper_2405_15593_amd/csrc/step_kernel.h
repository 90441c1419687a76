// The fused MicroAdam step: every stage of Algorithm 1 for a Top-K block in
// one workgroup of 256 threads, for blocks of 2049 to 4096 elements.  A
// workgroup takes BPW consecutive blocks and issues the loads of the next
// block before it works on the current one, so that its memory traffic
// continues through the select and the rebuild.
//
// Thread tid owns the 16 consecutive elements [16*tid, 16*tid + 16) of a
// block; its loads are the EF codes and bucket pairs, gradient, parameters
// and its share of the live window rows written at earlier steps.  Then:
//   1. a = g + Q^-1(e) in registers (Algorithm 1; Algorithm 2, Q^-1); a copy
//      goes to LDS, with the maximum |a| of every 8-element vector;
//   2. wave 0 finds the block Top-K of |a| (Section 3.1) from LDS in the
//      select kernel's three stages (a lower bound from half-lane maxima,
//      candidate compaction, a ballot search that stops early), assembles
//      the new window row (I, V) in element order and writes it as whole
//      128-byte lines (Section 3.2); where a stage overflows, all four waves
//      run an exact bitwise search instead, one barrier per bit;
//   3. every thread zeroes its kept elements and re-quantizes its residual:
//      bucket (min, max) and codes (Algorithm 1; Algorithm 2, Q; Lemma 1
//      with randomized rounding);
//   4. the live rows (the earlier ones as loaded, the new one from LDS) are
//      staged in LDS, oldest first.  Wave w owns the block's elements
//      [1024w, 1024w + 1024) (its threads' elements): it finds each row's
//      entries in that range (rows are in element order) and adds them into
//      an LDS accumulator, row after row, oldest first -- sum beta1^r V, read
//      back by each thread for its elements, then sum beta2^r V^2 (Algorithm
//      2, AdamStats).  Waves touch disjoint words and a wave's LDS accesses
//      execute in order, so this needs no barrier;
//   5. every thread turns its elements' sums into the update theta <- (1 -
//      eta*lambda) theta - eta m/(eps + sqrt(v)) (Algorithm 1; Algorithm 4).
// The new row never makes a round trip through HBM, and the step is one
// launch over all blocks of all tensors.
//
// LDS: a (then the accumulator) 16.4 KB, the select's vectors and candidates
// 4.5 KB, the new row's lines, the staged entries, control words: 26.5 KB
// with bf16 window values.  The host takes this path for rows of at most 128
// entries whose live rows fit 16 chunks of 64.
#pragma once

#include "microadam_common.h"

namespace microadam {
namespace {

constexpr int kStepThreads = 256;
constexpr int kStepCap = kStepThreads * kLaneElems;  // 4096 elements
constexpr int kStepMaxK = 2 * kWave;                  // entries per row
constexpr int kStepChunks = 16;                       // staged chunks of 64 entries
constexpr int kStepRowWords = kStepMaxK * 2 + 64;     // the new row and its two edge lines
constexpr int kStepCtl = 32;                          // control words
#ifndef MICROADAM_STEP_BLOCKS
#define MICROADAM_STEP_BLOCKS 1
#endif
constexpr int kStepBlocks = MICROADAM_STEP_BLOCKS;    // consecutive blocks per workgroup

template <bool VF>
__host__ __device__ constexpr size_t step_kernel_lds_words() {
  return (size_t)(kStepCap + 16) + kStepCap / 8 + kMaxCandVec + 2 * kCandMax + kStepRowWords +
         (size_t)kStepChunks * kWave * (VF ? 2 : 1) + kStepCtl;
}

// Word of element i in the accumulator: each thread's 16 elements are four
// 16-byte words at a stride of 4*NT words, so that a wave's 16-byte accesses
// fall on consecutive addresses.
__device__ __forceinline__ uint32_t step_zpos(uint32_t i) {
  return ((i >> 2) & 3u) * (4u * kStepThreads) + (i >> 4) * 4u + (i & 3u);
}

// One thread's inputs for one block, loaded ahead of the block's processing.
template <bool LB, bool BF16, bool VF32, int EFM>
struct StepIn {
  static constexpr int NP = kStepChunks * kWave / kStepThreads;  // staged positions per thread
  LaneIn<kLaneElems, LB, BF16, EFM> in;  // EF codes, bucket pairs, gradient
  Raw8<BF16> th[2];                       // parameters
  typename Entry<VF32>::T wv[NP];         // entries of the live rows written at earlier steps
  uint32_t edge_old;                      // wave 0: a word of the new row's first or last line
};

// Where the new row of block gb lies in its window record: bytes [row_lo,
// row_hi), inside the whole 128-byte lines [span_lo, span_hi).
struct RowSpan {
  uint32_t row_lo, row_hi, span_lo, span_hi, edge_off;
};

template <bool VF32>
__device__ __forceinline__ RowSpan row_span(const StepParams& p, int kq, int lane) {
  constexpr uint32_t EB = VF32 ? 8u : 4u;
  RowSpan r;
  r.row_lo = (uint32_t)p.new_slot * (uint32_t)kq * EB;
  r.row_hi = r.row_lo + (uint32_t)kq * EB;
  r.span_lo = r.row_lo & ~127u;
  r.span_hi = (r.row_hi + 127u) & ~127u;
  r.edge_off = lane < 32 ? r.span_lo + 4 * lane : r.span_hi - 128 + 4 * (lane - 32);
  return r;
}

// Issues every load of block gb for thread tid.
template <bool LB, bool BF16, bool VF32, int EFM>
__device__ __forceinline__ void step_load(const StepParams& p, int64_t gb, int tid, StepIn<LB, BF16, VF32, EFM>& x) {
  using E = Entry<VF32>;
  constexpr int NT = kStepThreads, NP = StepIn<LB, BF16, VF32, EFM>::NP;
  const int lane = tid & (kWave - 1);
  const uint32_t eb = (uint32_t)tid * kLaneElems;
  const int bl = p.bucket_log2;
  const uint32_t nbk = (uint32_t)(p.block >> bl);
  const uint32_t ef_bytes = (EFM & kEf8) ? (uint32_t)p.block : (uint32_t)(p.block >> 1);
  const Rsrc re = make_rsrc(p.state + p.ef_plane + (uint64_t)gb * ef_bytes, ef_bytes);
  const Rsrc rs = make_rsrc(p.state + p.stats_plane + (uint64_t)gb * nbk * 8, nbk * 8);
  lane_load_state(x.in, re, rs, eb, bl, false);
  const Block b = locate(p, gb);
  const Rsrc rg = make_rsrc((const uint8_t*)b.desc.grad + b.e0 * (BF16 ? 2 : 4), vec_bytes<BF16>(b.s));
  lane_load_grad(x.in, rg, eb);
  const Rsrc rp = make_rsrc((const uint8_t*)b.desc.param + b.e0 * (BF16 ? 2 : 4), vec_bytes<BF16>(b.s));
#pragma unroll
  for (int v = 0; v < 2; ++v) x.th[v] = load8<BF16>(rp, eb + 8 * v);
  // The live rows in the order the rebuild adds them, oldest first: chunk c
  // is part c mod R of live row c / R (R = ceil(k/64) parts of 64 entries,
  // 1 or 2).  Rows written at earlier steps are loaded here; the newest row
  // (the last live one) comes from LDS once the select has made it.
  const int kq = b.kq, m = p.window, n_live = p.n_live;
  const int slot0 = (p.new_slot + 1 + m - n_live) % m;  // the row written at step s is slot (s-1) mod m
  const int R = kq > kWave ? 2 : 1;
  const Rsrc rw = window_rsrc<VF32 ? 2 : 1>(p, gb, kq);
#pragma unroll
  for (int i = 0; i < NP; ++i) {
    const int q = tid + NT * i, c = q >> 6;
    const int row = R == 1 ? c : c >> 1;
    const int jj = (c - row * R) * kWave + (q & (kWave - 1));
    int slot = slot0 + row;
    if (slot >= m) slot -= m;
    x.wv[i] = E::none();
    if (row < n_live - 1 && jj < kq) x.wv[i] = E::load(rw, (uint32_t)(slot * kq + jj));
  }
  // The new row is written as the whole lines that cover it (records are
  // whole lines): wave 0 reads the words of the first and last line that lie
  // outside the row, to write them back unchanged.
  x.edge_old = 0;
  if (tid < kWave) {
    const RowSpan sp = row_span<VF32>(p, kq, lane);
    const Rsrc rrec = make_rsrc(p.state + p.win_plane + (uint64_t)gb * p.win_stride, (uint32_t)p.win_stride);
    x.edge_old = __builtin_amdgcn_raw_buffer_load_b32(rrec, sp.edge_off, 0, 0);
  }
}

// Every stage of the step for block gb, from the thread's loaded inputs.
template <bool LB, bool BF16, bool VF32, int EFM>
__device__ __forceinline__ void step_process(const StepParams& p, int64_t gb, int tid,
                                             StepIn<LB, BF16, VF32, EFM>& x, uint32_t* smem) {
  constexpr int NT = kStepThreads, NW = NT / kWave, CAP = kStepCap;
  constexpr int NVS = CAP / kWave / 8;  // vectors of 8 per lane in wave 0's view of the block
  constexpr int NP = StepIn<LB, BF16, VF32, EFM>::NP;
  constexpr uint32_t EB = VF32 ? 8u : 4u;
  using E = Entry<VF32>;
  using ET = typename E::T;
  static_assert(NVS == 8, "wave 0 holds 64 elements per lane");
  float* const za = (float*)smem;                        // [CAP + 16]: a, then the accumulator
  float* const vm = za + CAP + 16;                       // [CAP / 8] vector maxima
  uint32_t* const regi = (uint32_t*)(vm + CAP / 8);      // [kMaxCandVec] candidate vectors
  float* const cval = (float*)(regi + kMaxCandVec);      // [kCandMax] candidate values
  uint32_t* const cidx = (uint32_t*)(cval + kCandMax);   // [kCandMax] candidate indices
  uint32_t* const rowbuf = cidx + kCandMax;              // [kStepRowWords] the new row's lines
  ET* const stage = (ET*)(rowbuf + kStepRowWords);       // [kStepChunks * 64] staged entries
  uint32_t* const ctl = (uint32_t*)(stage + kStepChunks * kWave);  // [kStepCtl]
  // ctl: [0] T, [1] notie | general << 1, [2] i_last, [4, 12) per-wave sums
  // (two buffers), [12, 20) per-wave scan totals (two slots), [20] the index
  // of the last kept key equal to T

  const int lane = tid & (kWave - 1), wave = (int)sgpr((uint32_t)tid / kWave);
  const uint32_t eb = (uint32_t)tid * kLaneElems;
  const int bl = p.bucket_log2;
  if (tid == 0) ctl[20] = 0u;
  const uint32_t nbk = (uint32_t)(p.block >> bl);
  const uint32_t ef_bytes = (EFM & kEf8) ? (uint32_t)p.block : (uint32_t)(p.block >> 1);
  const Rsrc re = make_rsrc(p.state + p.ef_plane + (uint64_t)gb * ef_bytes, ef_bytes);
  const Rsrc rs = make_rsrc(p.state + p.stats_plane + (uint64_t)gb * nbk * 8, nbk * 8);
  const Block b = locate(p, gb);
  const int s = b.s, kq = b.kq;
  const bool full = s == CAP;
  const Rsrc rp = make_rsrc((const uint8_t*)b.desc.param + b.e0 * (BF16 ? 2 : 4), vec_bytes<BF16>(s));
  const int m = p.window, n_live = p.n_live;
  const int R = kq > kWave ? 2 : 1;
  const int nch = n_live * R;
  const RowSpan sp = row_span<VF32>(p, kq, lane);
  const uint32_t row_lo = sp.row_lo, row_hi = sp.row_hi, span_lo = sp.span_lo, span_hi = sp.span_hi;
  const uint32_t edge_off = sp.edge_off;
  const uint32_t row_w0 = (row_lo - span_lo) >> 2;  // rowbuf word of entry 0
  const Rsrc rrec = make_rsrc(p.state + p.win_plane + (uint64_t)gb * p.win_stride, (uint32_t)p.win_stride);
  (void)m;

  // ---------------------------------------------- 1. a = g + Q^-1(e)
  float a[2][8];
  const int rem = s - (int)eb;  // this thread's elements below the end of the block: [0, rem)
  lane_decode(x.in, a, rem, full);
  {
    float vmax[2];
    lane_vmax<kLaneElems>(a, vmax);
#pragma unroll
    for (int q = 0; q < 4; ++q)
      *(float4*)(za + q * 4 * NT + tid * 4) =
          make_float4(a[q >> 1][4 * (q & 1)], a[q >> 1][4 * (q & 1) + 1], a[q >> 1][4 * (q & 1) + 2],
                      a[q >> 1][4 * (q & 1) + 3]);
    *(float2*)(vm + 2 * tid) = make_float2(vmax[0], vmax[1]);
  }
  lds_sync();

  // ---------------------------------------------- 2. Top-K (wave 0)
  if (wave == 0) {
    // lane l's view: the 64 elements [64l, 64l + 64), vectors [8l, 8l + 8)
    const uint32_t le = (uint32_t)lane * 64;
    float vx[NVS];
    {
      const float4 x0 = *(const float4*)(vm + NVS * lane), x1 = *(const float4*)(vm + NVS * lane + 4);
      vx[0] = x0.x; vx[1] = x0.y; vx[2] = x0.z; vx[3] = x0.w;
      vx[4] = x1.x; vx[5] = x1.y; vx[6] = x1.z; vx[7] = x1.w;
    }
    uint32_t T = 0, i_last = 0;
    bool notie = false;
    bool general = kq > 2 * kWave;
    if (!general) {
      // stage 1: a lower bound L of the k-th largest |a|: the largest 13-bit
      // prefix with at least k of the 128 half-lane maxima at or above it
      float h0 = vx[0], h1 = vx[NVS / 2];
#pragma unroll
      for (int v = 1; v < NVS / 2; ++v) {
        h0 = __builtin_fmaxf(h0, vx[v]);
        h1 = __builtin_fmaxf(h1, vx[NVS / 2 + v]);
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
      // stage 2a: the vectors holding an element >= L, in element order
      bool f[NVS];
      uint32_t cnt = 0;
#pragma unroll
      for (int v = 0; v < NVS; ++v) {
        f[v] = vx[v] >= L;
        cnt += f[v] ? 1u : 0u;
      }
      uint32_t nvec;
      const uint32_t pre = lane_prefix(cnt, nvec);
      general = Lb == 0 || nvec > (uint32_t)kMaxCandVec;
      if (!general) {
        {
          uint32_t pos = pre;
#pragma unroll
          for (int v = 0; v < NVS; ++v)
            if (f[v]) regi[pos++] = le + 8 * v;
        }
        wave_sync();
        // stage 2b: the elements >= L of candidate vectors lane and lane + 64
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
            const uint32_t src = have ? regi[j] : 0u;
            const float4 x0 = *(const float4*)(za + step_zpos(src));
            const float4 x1 = *(const float4*)(za + step_zpos(src + 4));
            cb[r] = src;
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
          // stage 3: the k-th largest key among the C candidates, bit by bit
          // from the top; it stops once exactly k candidates are at or above
          // the prefix (below L the candidate count is not the block's)
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
                const uint32_t w = row_w0 + (sel_before + lanes_below(sm)) * (EB / 4);
                const ET x = E::make(ci[r], cf[r]);
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
          if (edge_off < row_lo || edge_off >= row_hi) rowbuf[(edge_off - span_lo) >> 2] = x.edge_old;
          wave_sync();
          const uint32_t nvec4 = (span_hi - span_lo) >> 4;
          for (uint32_t q = (uint32_t)lane; q < nvec4; q += kWave)
            __builtin_amdgcn_raw_buffer_store_b128(*(const u32x4*)(rowbuf + 4 * q), rrec, span_lo + 16 * q, 0, 0);
        }
      }
    }
    if (lane == 0) {
      ctl[0] = T;
      ctl[1] = (notie ? 1u : 0u) | (general ? 2u : 0u);
      ctl[2] = i_last;
    }
  }
  lds_sync();
  uint32_t T = sgpr(ctl[0]), i_last = sgpr(ctl[2]);
  const uint32_t flags = sgpr(ctl[1]);
  bool notie = (flags & 1u) != 0;

  if (flags & 2u) {
    // Exact bitwise search over the whole block by all waves (ties at the
    // threshold, candidates overflowing LDS): the largest T with #{|a| >=
    // T} >= k, one barrier per bit.  |a| is compared against the float with
    // the same bits (the order of the keys for finite values).
    auto wg_sum = [&](uint32_t wave_value, int buf) {
      if (lane == 0) ctl[4 + buf * NW + wave] = wave_value;
      lds_sync();
      uint32_t t = 0;
#pragma unroll
      for (int w = 0; w < NW; ++w) t += ctl[4 + buf * NW + w];
      return sgpr(t);
    };
    // exclusive prefix in element order of a per-thread count below 32, and
    // the workgroup total
    auto wg_scan = [&](uint32_t c, int slot, uint32_t& total) {
      uint32_t in_wave = 0, wave_total = 0;
#pragma unroll
      for (int b2 = 0; b2 < 5; ++b2) {
        const uint64_t mk = ballot((c >> b2) & 1u);
        in_wave += lanes_below(mk) << b2;
        wave_total += popc(mk) << b2;
      }
      if (lane == 0) ctl[12 + slot * NW + wave] = wave_total;
      lds_sync();
      uint32_t before = 0, all = 0;
#pragma unroll
      for (int w = 0; w < NW; ++w) {
        const uint32_t x = ctl[12 + slot * NW + w];
        all += x;
        before += w < wave ? x : 0u;
      }
      total = sgpr(all);
      return sgpr(before) + in_wave;
    };
    uint32_t t = 0;
    bool exact = false;
    int buf = 0;
    for (int bit = 30; bit >= 0 && !exact; --bit) {
      const uint32_t c = t | (1u << bit);
      const float cf = __uint_as_float(c);
      uint32_t n = 0;
#pragma unroll
      for (int v = 0; v < 2; ++v)
#pragma unroll
        for (int e = 0; e < 8; ++e) n += popc(ballot(__builtin_fabsf(a[v][e]) >= cf));
      n = wg_sum(n, buf);
      buf ^= 1;
      if (n >= (uint32_t)kq) {
        t = c;
        exact = n == (uint32_t)kq;
      }
    }
    T = t;
    uint32_t sel_l = 0;
    const float tf = opaque_f(__uint_as_float(t));
    if (exact) {
      notie = true;
#pragma unroll
      for (int v = 0; v < 2; ++v)
#pragma unroll
        for (int e = 0; e < 8; ++e) sel_l += __builtin_fabsf(a[v][e]) >= tf ? 1u : 0u;
    } else {
      // the keys above t are kept, then the first `need` keys equal to t in
      // element order
      uint32_t ngt_l = 0, neq_l = 0;
#pragma unroll
      for (int v = 0; v < 2; ++v)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          ngt_l += __builtin_fabsf(a[v][e]) > tf ? 1u : 0u;
          neq_l += __builtin_fabsf(a[v][e]) == tf ? 1u : 0u;
        }
      uint32_t ngt_w = 0;
#pragma unroll
      for (int b2 = 0; b2 < 5; ++b2) ngt_w += popc(ballot((ngt_l >> b2) & 1u)) << b2;
      const uint32_t need = (uint32_t)kq - wg_sum(ngt_w, buf);  // >= 1
      uint32_t neq_all;
      const uint32_t eq_pre = wg_scan(neq_l, 0, neq_all);
      // the thread holding the need-th key equal to t (with finite keys
      // exactly one; a NaN reaches no threshold, and ctl[20] then keeps 0)
      if (eq_pre < need && eq_pre + neq_l >= need) {
        const float tf2 = opaque_f(tf);
        uint32_t r = eq_pre, my_last = 0;
#pragma unroll
        for (int v = 0; v < 2; ++v)
#pragma unroll
          for (int e = 0; e < 8; ++e)
            if (__builtin_fabsf(a[v][e]) == tf2) {
              if (r == need - 1) my_last = eb + 8 * v + e;
              ++r;
            }
        ctl[20] = my_last;
      }
      lds_sync();
      i_last = sgpr(ctl[20]);
      notie = neq_all == need;
      const int last_here = (int)i_last - (int)eb;
      const float tf3 = opaque_f(tf);
#pragma unroll
      for (int v = 0; v < 2; ++v)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float ab = __builtin_fabsf(a[v][e]);
          sel_l += ((ab > tf3) | ((ab == tf3) & (8 * v + e <= last_here))) ? 1u : 0u;
        }
    }
    // the new row in element order, into LDS (positions past the row's k
    // entries are never written), then wave 0 writes its lines
    uint32_t kept_all;
    uint32_t pos = wg_scan(sel_l, 1, kept_all);
    if (sel_l) {
      const float tf4 = opaque_f(tf);
      const int last_here = notie ? CAP : (int)i_last - (int)eb;
#pragma unroll
      for (int v = 0; v < 2; ++v)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float ab = __builtin_fabsf(a[v][e]);
          if ((ab > tf4) | ((ab == tf4) & (8 * v + e <= last_here))) {
            if (pos < (uint32_t)kq) {
              const ET x = E::make(eb + 8 * v + e, a[v][e]);
              if constexpr (VF32) *(u32x2*)(rowbuf + row_w0 + 2 * pos) = x;
              else rowbuf[row_w0 + pos] = x;
            }
            ++pos;
          }
        }
    }
    lds_sync();
    if (wave == 0) {
      if (edge_off < row_lo || edge_off >= row_hi) rowbuf[(edge_off - span_lo) >> 2] = x.edge_old;
      wave_sync();
      const uint32_t nvec4 = (span_hi - span_lo) >> 4;
      for (uint32_t q = (uint32_t)lane; q < nvec4; q += kWave)
        __builtin_amdgcn_raw_buffer_store_b128(*(const u32x4*)(rowbuf + 4 * q), rrec, span_lo + 16 * q, 0, 0);
    }
  }

  // ---------------------------------------------- 3. e = Q(a with a[I] = 0)
  lane_quantize_store<kLaneElems, LB, EFM>(a, T, notie, i_last, eb, s, rem, full, bl, false, re, rs,
                                           EfStream{b.e0, b.j, (uint32_t)p.t, p.seed_lo, p.seed_hi});

  // ---------------------------------------------- 4. moments from the window
  // The live rows' entries as they are (index | value), oldest first; every
  // thread clears its own accumulator words.
#pragma unroll
  for (int i = 0; i < NP; ++i) {
    const int q = tid + NT * i, c = q >> 6;
    const int row = R == 1 ? c : c >> 1;
    const int jj = (c - row * R) * kWave + (q & (kWave - 1));
    ET e = x.wv[i];
    if (row == n_live - 1 && jj < kq) {
      if constexpr (VF32) e = *(const u32x2*)(rowbuf + row_w0 + 2 * jj);
      else e = rowbuf[row_w0 + jj];
    }
    if (c >= nch || jj >= kq) e = E::none();
    stage[q] = e;
  }
  {
    const float4 zero = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int q = 0; q < 4; ++q) *(float4*)(za + q * 4 * NT + tid * 4) = zero;
  }
  lds_sync();
  // Wave w adds the entries of its elements [1024w, 1024w + 1024).  Lane r <
  // n_live finds where live row r's entries reach 1024w, lane 32 + r where
  // they reach 1024(w + 1): binary searches over the row, whose entries are
  // in ascending index order (unused positions hold kNoEntry, above all).
  uint32_t bound = 0;
  {
    const int r = lane & 31;
    if (r < n_live) {
      const uint32_t key = 1024u * (uint32_t)wave + (lane >= 32 ? 1024u : 0u);
      const ET* const rw_lds = stage + r * kWave * R;
      uint32_t lo = 0, n = (uint32_t)kq;
      while (n > 0) {
        const uint32_t half = n >> 1;
        if (E::idx(rw_lds[lo + half]) < key) {
          lo += half + 1;
          n -= half + 1;
        } else {
          n = half;
        }
      }
      bound = lo;
    }
  }
  const float w1s = lane < kMaxWindow ? constant_ptr(p.wpow)[lane] : 0.0f;
  const float w2s = lane < kMaxWindow ? constant_ptr(p.wpow)[kMaxWindow + lane] : 0.0f;
  // the longest of the wave's row segments (uniform)
  uint32_t seg_max = 0;
#pragma unroll
  for (int r = 0; r < kStepChunks; ++r) {
    if (r < n_live) {
      const uint32_t len = __builtin_amdgcn_readlane(bound, 32 + r) - __builtin_amdgcn_readlane(bound, r);
      seg_max = len > seg_max ? len : seg_max;
    }
  }
  float s1[16], s2[16];
  // this thread's accumulator words, then cleared (the wave's own LDS
  // accesses are ordered, and no other wave touches these words)
  auto take = [&](float (&out)[16], bool clear) {
    wave_sync();
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const float4 u = *(const float4*)(za + q * 4 * NT + tid * 4);
      out[4 * q] = u.x; out[4 * q + 1] = u.y; out[4 * q + 2] = u.z; out[4 * q + 3] = u.w;
      if (clear) *(float4*)(za + q * 4 * NT + tid * 4) = make_float4(0.f, 0.f, 0.f, 0.f);
    }
  };
  auto weight = [&](float ws, int r) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(ws), n_live - 1 - r));
  };
  if (seg_max <= (uint32_t)kWave) {
    // every row holds at most 64 entries of the wave's elements: lane j
    // takes entry j of each row's segment, all rows loaded at once
    ET xr[kStepChunks];
#pragma unroll
    for (int r = 0; r < kStepChunks; ++r) {
      xr[r] = E::none();
      if (r < n_live) {
        const uint32_t lo = __builtin_amdgcn_readlane(bound, r), hi = __builtin_amdgcn_readlane(bound, 32 + r);
        if (lo + lane < hi) xr[r] = stage[r * kWave * R + lo + lane];
      }
    }
    auto add_rows = [&](bool second) {
#pragma unroll
      for (int r = 0; r < kStepChunks; ++r) {
        if (r < n_live) {
          const uint32_t i = E::idx(xr[r]);
          if (i < (uint32_t)s) {
            const uint32_t zw = step_zpos(i);
            const float v = E::val(xr[r]);
            const float t = second ? weight(w2s, r) * (v * v) : weight(w1s, r) * v;
            const float acc = za[zw];
            za[zw] = acc + t;
          }
        }
      }
    };
    add_rows(false);
    take(s1, true);
    add_rows(true);
    take(s2, false);
  } else {
    // longer segments: 64 entries of a row at a time
    auto add_rows = [&](bool second) {
      for (int r = 0; r < n_live; ++r) {
        const uint32_t lo = __builtin_amdgcn_readlane(bound, r), hi = __builtin_amdgcn_readlane(bound, 32 + r);
        const float w = second ? weight(w2s, r) : weight(w1s, r);
        for (uint32_t j = lo + lane; j < hi; j += kWave) {
          const ET e = stage[r * kWave * R + j];
          const uint32_t i = E::idx(e);
          if (i < (uint32_t)s) {
            const uint32_t zw = step_zpos(i);
            const float v = E::val(e);
            const float acc = za[zw];
            za[zw] = acc + (second ? w * (v * v) : w * v);
          }
        }
      }
    };
    add_rows(false);
    take(s1, true);
    add_rows(true);
    take(s2, false);
  }

  // ---------------------------------------------- 5. parameter update
  // (an element without window entries has both sums 0 and keeps theta,
  // less the decay)
#pragma unroll
  for (int v = 0; v < 2; ++v) {
    float thf[8], out[8];
    unpack8<BF16>(x.th[v], thf);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float a1 = s1[8 * v + e], a2 = s2[8 * v + e];
      const bool none = (a1 == 0.0f) & (a2 == 0.0f);
      const float mh = p.c1 * a1, vh = p.c2 * a2;
      // correctly rounded square root and division
      const float d = none ? 0.0f : p.lr * (mh / (p.eps + __builtin_sqrtf(vh)));
      const float base = thf[e] * p.decay;  // exact when the factor is 1
      out[e] = base - d;
    }
    store8<BF16>(rp, eb + 8 * v, s, full, out);
  }
}

template <bool LB, bool BF16, bool VF32, int EFM, int BPW>
__global__ void __launch_bounds__(kStepThreads)
__attribute__((amdgpu_waves_per_eu(BPW > 1 ? 4 : VF32 ? 5 : 6)))
step_kernel(StepParams p, int64_t first, int64_t count) {
  extern __shared__ __align__(16) uint32_t smem[];
  const int tid = thread_id();
  // workgroup w takes the BPW consecutive blocks of group xcd_block(w)
  const int64_t groups = (count + BPW - 1) / BPW;
  const int64_t g0 = first + xcd_block(block_id(), groups) * BPW, end = first + count;
  StepIn<LB, BF16, VF32, EFM> cur, nxt;
  step_load(p, g0, tid, cur);
#pragma unroll
  for (int it = 0; it < BPW; ++it) {
    const int64_t gb = g0 + it;
    if (gb >= end) break;
    if (it + 1 < BPW && gb + 1 < end) step_load(p, gb + 1, tid, nxt);
    step_process(p, gb, tid, cur, smem);
    if (it + 1 < BPW) {
      cur = nxt;
      lds_sync();  // the next block reuses the LDS
    }
  }
}

// Blocks [first, first + count) of 2049 to 4096 elements, error-feedback
// format EFM; parameters and gradients of one dtype.
template <int EFM>
hipError_t launch_step_mode(const StepParams& p, int bf16, int value_f32, int64_t first, int64_t count,
                            hipStream_t stream) {
  if (count <= 0) return hipSuccess;
  const dim3 threads(kStepThreads);
  const bool lb = (1 << p.bucket_log2) >= kLaneElems;
  auto go = [&](auto lb_tag, auto bf_tag, auto vf_tag) {
    constexpr bool LB = decltype(lb_tag)::value, BF = decltype(bf_tag)::value, VF = decltype(vf_tag)::value;
    const dim3 groups((uint32_t)((count + kStepBlocks - 1) / kStepBlocks));
    hipLaunchKernelGGL((step_kernel<LB, BF, VF, EFM, kStepBlocks>), groups, threads, step_kernel_lds_words<VF>() * 4,
                       stream, p, first, count);
    return hipGetLastError();
  };
  using T = std::true_type;
  using F = std::false_type;
  if (lb) {
    if (bf16) return value_f32 ? go(T{}, T{}, T{}) : go(T{}, T{}, F{});
    return value_f32 ? go(T{}, F{}, T{}) : go(T{}, F{}, F{});
  }
  if (bf16) return value_f32 ? go(F{}, T{}, T{}) : go(F{}, T{}, F{});
  return value_f32 ? go(F{}, F{}, T{}) : go(F{}, F{}, F{});
}

}  // namespace
}  // namespace microadam
