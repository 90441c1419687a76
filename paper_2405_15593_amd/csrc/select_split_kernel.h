// The select for Top-K blocks above 4096 elements whose size is a multiple of
// 4096 (buckets inside blocks), in launches that stream a block instead of
// holding it: the threshold kernel finds each block's k-th largest |a| and
// the row position of each 4096-element sub-block's first kept entry; the
// apply kernel then runs one wave per sub-block (as the one-wave select does
// per block): it keeps the elements at or above the threshold, writes its
// part of the new row and of the segment table, and quantizes.  Blocks whose
// threshold search needs more than the streamed bracket (see below) are
// marked, skipped by the apply kernel and taken by the multi-wave select
// kernel, which holds the block and searches it exactly.
//
// The multi-wave kernel fills a compute unit's registers with one block, so
// a compute unit loads one block, then searches it with no loads in flight;
// the two streamed passes read the gradient and codes twice (2.56 B per
// parameter more) but keep loads in flight on every compute unit.
#pragma once

#include "microadam_common.h"

namespace microadam {
namespace {

constexpr int kThrThreads = 256;                   // threshold kernel: four waves per block
constexpr int kThrWaves = kThrThreads / kWave;
constexpr int kThrSamples = 1024;                  // sample keys (128 vectors of 8)
constexpr int kThrList = 1024;                     // bracketed keys gathered per wave
constexpr int kThrListStride = kThrList + kWave;   // + one sink slot per lane
constexpr int kThrSampleRes = 15;                  // the sample's order statistics to 2^15 (1/256 binade)
constexpr uint32_t kThrRecordBytes = 128;          // per block
constexpr uint32_t kAllTies = 0xFFFFFFFFu;         // i_last: every key equal to T is kept
constexpr uint32_t kApplyValWords = 2048;          // apply kernel: a sub-block's values as bf16
constexpr uint32_t kApplyStageWords = 448;         // apply kernel: row words staged in LDS

// LDS of an apply wave: the exchange and the codes' store of the one-wave
// select, then (bf16 entries) the sub-block's values and the staged row
constexpr size_t apply_lds_words() {
  return select_lds_words() > kApplyValWords + kApplyStageWords ? select_lds_words()
                                                                 : kApplyValWords + kApplyStageWords;
}
static_assert(16 * apply_lds_words() * 4 <= 163840, "sixteen apply waves fit a compute unit's LDS");

// The per-block record the threshold kernel writes (uint32 words):
//   [0] 1 when the bracket held the threshold (else the multi-wave select
//       takes the block), [1] T, the k-th largest key (|a| as an integer),
//   [2] i_last: keys equal to T are kept up to this block element (kAllTies:
//       all of them), [4 + w] the row position of sub-block w's first kept
//       entry (at most k_q).  Kept: key > T, or key == T and index <= i_last.
// (the sample is read into registers before the pass, which then
// overwrites it with gathered keys)
struct ThrLds {
  static constexpr int kSample = 0;                                  // [kThrSamples]
  static constexpr int kKeys = 0;                                    // [waves][kThrListStride] keys
  static constexpr int kIdx = kKeys + kThrWaves * kThrListStride;    // [waves][kThrListStride] uint16 indices
  static constexpr int kHi = kIdx + kThrWaves * kThrListStride / 2;  // [16] keys >= hi per sub-block
  static constexpr int kKept = kHi + 16;                             // [16] kept gathered keys per sub-block
  static constexpr int kCnt = kKept + 16;                            // [2][waves] per-wave counts
  static constexpr int kDig = kCnt + 2 * kThrWaves;                  // [2][32] digit counts
  static constexpr int kMisc = kDig + 64;                            // [4]
  static constexpr int kWords = kMisc + 4;
};
static_assert(1024 + kMaxBlock / 32 <= kThrWaves * kThrListStride, "histograms and bitmap fit the key lists");
static_assert(6 * ThrLds::kWords * 4 <= 163840, "six threshold workgroups fit a compute unit's LDS");

// One 8-element vector of the block: gradient, codes and bucket pair.
template <bool GBF16, int EFM>
struct VecIn {
  Raw8<GBF16> g;
  uint32_t c[(EFM & kEf8) ? 2 : 1];
  u32x2 st;
};

template <bool GBF16, int EFM>
__device__ __forceinline__ void vec_load(VecIn<GBF16, EFM>& x, Rsrc rg, Rsrc re, Rsrc rs, uint32_t j, int bl) {
  x.g.w[0] = __builtin_amdgcn_raw_buffer_load_b128(rg, j * (GBF16 ? 16u : 32u), 0, kStream);
  if constexpr (!GBF16) x.g.w[1] = __builtin_amdgcn_raw_buffer_load_b128(rg, j * 32u + 16u, 0, kStream);
  if constexpr (EFM & kEf8) {
    const u32x2 t = __builtin_amdgcn_raw_buffer_load_b64(re, j * 8u, 0, kStream);
    x.c[0] = t[0];
    x.c[1] = t[1];
  } else {
    x.c[0] = __builtin_amdgcn_raw_buffer_load_b32(re, j * 4u, 0, kStream);
  }
  x.st = __builtin_amdgcn_raw_buffer_load_b64(rs, ((8u * j) >> bl) * 8u, 0, kStream);
}

// a = g + Q^-1(e) of vector j (the arithmetic of lane_decode); elements at
// or past s are 0 (`full`, workgroup-uniform: no element is).
template <bool GBF16, int EFM>
__device__ __forceinline__ void vec_decode(const VecIn<GBF16, EFM>& x, uint32_t j, int s, bool full,
                                           float (&a)[8]) {
  const float lo = __uint_as_float(x.st[0]);
  const float u = ef_step<EFM>(__uint_as_float(x.st[1]) - lo);
  float g[8], c[8];
  unpack8<GBF16>(x.g, g);
  unpack_codes<EFM>(x.c, 0, c);
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float sc = c[e] * u;
    const float d = sc + lo;
    a[e] = g[e] + d;
  }
  if (!full) {
#pragma unroll
    for (int e = 0; e < 8; ++e)
      if ((int)(8 * j) + e >= s) a[e] = 0.0f;
  }
}

// ------------------------------------------------------ threshold kernel
// One 256-thread workgroup per block, in three parts.
//  1. A bracket [lo, hi) for the k-th largest key from 1024 sample keys (one
//     8-element vector out of every 128th of the block; vectors spread out,
//     since neighbouring elements share a bucket and so correlate): the
//     16-bit prefixes of the sample's order statistics three standard
//     deviations below and two above the expected rank, by a 16-ary search
//     (four digits per wave, one barrier per 4 bits).
//  2. One pass over the block, each wave's 1 KB vector loads contiguous:
//     keys >= hi are counted per sub-block, keys in [lo, hi) gathered with
//     their indices in the wave's part of LDS.  The bracket holds the answer
//     when fewer than k keys lie at or above hi, at least k at or above lo,
//     and no wave gathered more than kThrList; else the block is marked.
//  3. T by a radix select over the gathered keys (8 bits per round, an LDS
//     histogram per round), the ties at T kept in index order (the need-th
//     set bit of an LDS bitmap of their indices), and the row positions of
//     the sub-blocks from their kept counts.
// The bracket's rank arithmetic is approximate: the check in 2 decides.
// Six workgroups per compute unit (the LDS of ThrLds allows six, and the
// registers are held to 80 for it): measured 2.23-2.26 -> 2.02 ms for the
// select phase of the 1.5e9 workload against four workgroups with lists of
// 1536 keys; shorter lists overflow on that workload's ties.
template <bool GBF16, int EFM>
__global__ void __launch_bounds__(kThrThreads) __attribute__((amdgpu_waves_per_eu(6)))
threshold_kernel(StepParams p, int64_t first, int64_t count) {
  extern __shared__ __align__(16) uint32_t smem[];
  uint32_t* const samp = smem + ThrLds::kSample;
  uint32_t* const lkey = smem + ThrLds::kKeys;
  uint16_t* const lidx = (uint16_t*)(smem + ThrLds::kIdx);
  uint32_t* const hi_sb = smem + ThrLds::kHi;
  uint32_t* const kept_sb = smem + ThrLds::kKept;
  uint32_t* const cnt = smem + ThrLds::kCnt;
  uint32_t* const dig = smem + ThrLds::kDig;
  uint32_t* const misc = smem + ThrLds::kMisc;

  const int tid = thread_id(), lane = tid & (kWave - 1), wave = (int)sgpr((uint32_t)tid / kWave);
  const int64_t gb = first + xcd_block(block_id(), count);
  const Block b = locate(p, gb);
  const int s = b.s, kq = b.kq, bl = p.bucket_log2;
  const bool full = s == p.block;
  const uint32_t nvec = (uint32_t)p.block / 8;
  const uint32_t ef_bytes = (EFM & kEf8) ? (uint32_t)p.block : (uint32_t)p.block / 2;
  const uint32_t nbk = (uint32_t)(p.block >> bl);
  const Rsrc re = make_rsrc(p.state + p.ef_plane + (uint64_t)gb * ef_bytes, ef_bytes);
  const Rsrc rs = make_rsrc(p.state + p.stats_plane + (uint64_t)gb * nbk * 8, nbk * 8);
  const Rsrc rg = make_rsrc((const uint8_t*)b.desc.grad + b.e0 * (GBF16 ? 2 : 4), vec_bytes<GBF16>(s));
  const Rsrc rrec = make_rsrc(p.thr + (uint64_t)gb * kThrRecordBytes, kThrRecordBytes);
  using VI = VecIn<GBF16, EFM>;

  if (tid < 32) hi_sb[tid] = 0u;  // with kept_sb

  // ---------------------------------------------- 1. the sample bracket
  {
    const uint32_t seg = nvec / (kThrSamples / 8);  // vectors per 128th of the block (>= 8)
    uint32_t valid = 0;
    if (tid < kThrSamples / 8) {
      const uint32_t j = (uint32_t)tid * seg + ((uint32_t)tid * 5u) % seg;
      VI x;
      vec_load(x, rg, re, rs, j, bl);
      float a[8];
      vec_decode(x, j, s, full, a);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const uint32_t k = key_of(a[e]);
        const bool in = (int)(8 * j) + e < s;
        samp[8 * tid + e] = in && k <= 0x7F800000u ? k : 0u;  // a NaN sample counts as 0
        valid += in ? 1u : 0u;
      }
    }
    uint32_t vw = 0;
#pragma unroll
    for (int b2 = 0; b2 < 4; ++b2) vw += popc(ballot((valid >> b2) & 1u)) << b2;
    if (lane == 0) cnt[wave] = vw;
  }
  lds_sync();
  uint32_t ns = 0;
#pragma unroll
  for (int w = 0; w < kThrWaves; ++w) ns += cnt[w];
  ns = sgpr(ns);
  // approximate ranks from the top: the answer's expected rank in the sample,
  // three standard deviations below it for lo and two above it for hi (keys
  // >= hi are only counted, so a narrower upper side gathers fewer keys;
  // measured on the 1.5e9 workload, 3 and 2 beat 3 and 3, 3 and 1.5, and 3.5
  // and 2 by 0.05-0.15 ms per step, with the failures included)
  const float mu = (float)ns * (float)kq * __builtin_amdgcn_rcpf((float)s);
  const float sd = __builtin_amdgcn_sqrtf(mu);
  const int r_lo = (int)__builtin_ceilf(mu + 3.0f * sd), r_hi = (int)__builtin_floorf(mu - 2.0f * sd);
  uint32_t lo, hi;
  {
    uint32_t key[kThrSamples / kWave];
#pragma unroll
    for (int j = 0; j < kThrSamples / kWave; ++j) key[j] = samp[lane + kWave * j];
    // tl, th: the largest 16-bit prefixes (bits 30..15) with at least r_lo,
    // r_hi sample keys at or above them; wave w counts digits 4w .. 4w + 3
    uint32_t tl = 0, th = 0;
#pragma unroll
    for (int rd = 0; rd < 4; ++rd) {
      const int sh = 27 - 4 * rd;
      uint32_t* const dg = dig + (rd & 1) * 32;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const uint32_t d = (uint32_t)(wave * 4 + i);
        if (d == 0) continue;
        const uint32_t cl = tl + (d << sh), ch = th + (d << sh);
        uint32_t nl = 0, nh = 0;
#pragma unroll
        for (int j = 0; j < kThrSamples / kWave; ++j) {
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
    lo = r_lo > (int)ns ? 1u : (tl > 1u ? tl : 1u);  // a key of 0 is never gathered
    hi = r_hi < 1 ? 1u << 31 : th + (1u << kThrSampleRes);
  }

  // ---------------------------------------------- 2. the streamed pass
  // The lanes of an element in the bracket append it (its a, whose sign
  // the reads below drop, and its index) to the wave's list; a vector whose
  // 512 elements might not fit the list's remaining room takes the checked
  // form, where positions past the list go to the lane's sink slot (the
  // count still grows: overflow is detected).
  const uint32_t vpt = nvec / kThrThreads;  // vectors per thread: even, 4 .. 32
  uint32_t* const mykey = lkey + wave * kThrListStride;
  uint16_t* const myidx = lidx + wave * kThrListStride;
  uint32_t wn = 0;  // keys this wave found in the bracket
  {
    const float lof = __uint_as_float(lo), hif = __uint_as_float(hi < 0x7F800000u ? hi : 0x7F800000u);
    auto pass = [&](auto nohi_tag) {
      constexpr bool NOHI = decltype(nohi_tag)::value;
      const float lob_u = opaque_f(lof), hib_u = opaque_f(hif);
      for (uint32_t r0 = 0; r0 < vpt; r0 += 8) {
        // (all eight loads go out unconditionally, so that none waits on
        // another; a vector past the block reads zeros through the buffer
        // bounds and is not used)
        VI x[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) vec_load(x[i], rg, re, rs, kThrThreads * (r0 + i) + kWave * wave + lane, bl);
        // the wave's keys >= hi in the round's four sub-blocks, counted from
        // the lane masks of the bracket test's two compares (>= lo and not
        // < hi, so that a NaN, which fails both, is not counted)
        uint32_t nh[4] = {0u, 0u, 0u, 0u};
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          if (r0 + i >= vpt) continue;
          const uint32_t j = kThrThreads * (r0 + i) + kWave * wave + lane;
          float a[8];
          vec_decode(x[i], j, s, full, a);
          auto gather = [&](auto checked_tag) {
            constexpr bool CHECKED = decltype(checked_tag)::value;
            // (the rare checked form compares against its own copies of the
            // bounds, so that the compiler does not hoist its compares above
            // the branch and then compute them again in the common form)
            const float lob = CHECKED ? opaque_f(lob_u) : lob_u, hib = CHECKED ? opaque_f(hib_u) : hib_u;
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              const float ab = __builtin_fabsf(a[e]);
              const bool ge_lo = ab >= lob, below = NOHI || ab < hib;
              const bool in = ge_lo & below;
              // (the masks from the compares themselves rather than from `in`)
              const uint64_t m_ge = ballot(ab >= lob);
              const uint64_t m_lt = NOHI ? ~0ull : ballot(ab < hib);
              if constexpr (!NOHI) nh[i >> 1] = sgpr(nh[i >> 1] + popc(m_ge & ~m_lt));
              const uint64_t mi = m_ge & m_lt;
              if constexpr (CHECKED) {
                const uint32_t pos = lanes_below_from(mi, wn);
                const uint32_t at = in && pos < (uint32_t)kThrList ? pos : (uint32_t)(kThrList + lane);
                mykey[at] = __float_as_uint(a[e]);
                myidx[at] = (uint16_t)(8 * j + e);
              } else if (in) {
                const uint32_t pos = lanes_below_from(mi, wn);
                mykey[pos] = __float_as_uint(a[e]);
                myidx[pos] = (uint16_t)(8 * j + e);
              }
              wn = sgpr(wn + popc(mi));
            }
          };
          if (sgpr(wn) + 8u * kWave <= (uint32_t)kThrList)
            gather(BoolTag<false>{});
          else
            gather(BoolTag<true>{});
          __builtin_amdgcn_sched_barrier(0);  // one vector at a time
        }
        if (!NOHI) {
#pragma unroll
          for (int q = 0; q < 4; ++q)
            if (lane == 0 && nh[q] != 0u) atomicAdd(&hi_sb[(r0 >> 1) + q], nh[q]);
        }
      }
    };
    if (hi > 0x7F800000u)
      pass(BoolTag<true>{});
    else
      pass(BoolTag<false>{});
  }
  if (lane == 0) cnt[kThrWaves + wave] = wn;
  lds_sync();
  uint32_t n_hi = 0, n_in = 0;
  bool over = false;
#pragma unroll
  for (int w = 0; w < kThrWaves; ++w) {
    const uint32_t c = cnt[kThrWaves + w];
    n_in += c;
    over |= c > (uint32_t)kThrList;
  }
  {
    const uint32_t h = lane < 16 ? hi_sb[lane] : 0u;
    uint32_t t = h;
#pragma unroll
    for (int d = 1; d < 16; d <<= 1) t += __shfl_xor(t, d, kWave);
    n_hi = sgpr(t);
  }
  n_in = sgpr(n_in);
  const bool ok = !over && lo <= 0x7F800000u && n_hi < (uint32_t)kq && n_hi + n_in >= (uint32_t)kq;
  if (!ok) {
    // the record says so, and the block joins the list the multi-wave select
    // works through
    if (tid == 0) {
      __builtin_amdgcn_raw_buffer_store_b32(0u, rrec, 0, 0, 0);
      uint32_t* const list = (uint32_t*)(p.thr + thr_list_offset(p.total_blocks));
      const uint32_t at = __hip_atomic_fetch_add(list, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (at < (uint64_t)p.total_blocks) list[4 + at] = (uint32_t)gb;
    }
    return;
  }

  // ---------------------------------------------- 3. T, the ties, the offsets
  // T is the kp-th largest gathered key (kp = k - n_hi), found by a radix
  // select over rel = key - lo (< hi - lo), 8 bits per round from the top
  // bit of hi - lo - 1: a 256-bin LDS histogram of the digit among the keys
  // still in play, then every wave picks the digit where the count from the
  // top reaches the keys still needed (one barrier per round; histograms
  // alternate, each cleared the round before its use).
  const uint32_t mine = sgpr(cnt[kThrWaves + wave]);  // <= kThrList
  constexpr int NR = kThrList / kWave;
  uint32_t y[NR];
#pragma unroll
  for (int r = 0; r < NR; ++r) {
    const uint32_t q = (uint32_t)(lane + kWave * r);
    y[r] = q < mine ? (mykey[q] & 0x7FFFFFFFu) - lo : 0xFFFFFFFFu;  // rel; past the list: out of play
  }
  // every wave holds its keys now: the key lists become the four rounds'
  // histograms and the tie bitmap, cleared before any use
  lds_sync();
  uint32_t* const hist = lkey;          // [4][256]
  uint32_t* const bits = lkey + 1024;   // [p.block / 32]
  const uint32_t nw32 = (uint32_t)p.block / 32u;
  for (uint32_t q = (uint32_t)tid; q < 1024u + nw32; q += kThrThreads) lkey[q] = 0u;
  lds_sync();
  const uint32_t width = hi - lo;
  const int nbits = 32 - __builtin_clz((width - 1u) | 1u);
  const uint32_t kp = (uint32_t)kq - n_hi;  // 1 <= kp <= n_in
  uint32_t pre = 0;                         // rel prefix chosen so far (its bits >= sh_prev)
  int sh_prev = 32;                         // 32: no prefix yet
  uint32_t above = 0;                       // gathered keys above the prefix's range
  uint32_t n_eq = 0;                        // gathered keys equal to T (the last round's bin)
  for (int rd = 0; sh_prev > 0; ++rd) {
    // the first round takes the top 1-8 bits of rel, the others 8 each
    const int sh = rd == 0 ? (nbits - 1) / 8 * 8 : sh_prev - 8;
    uint32_t* const h = hist + rd * 256;
#pragma unroll
    for (int r = 0; r < NR; ++r) {
      const uint32_t v = y[r];
      const bool play = v < width && (rd == 0 || (v >> sh_prev) == pre);
      if (play) atomicAdd(&h[(v >> sh) & 255u], 1u);
    }
    lds_sync();
    // digits 4l .. 4l + 3 in lane l; counts from the top
    const u32x4 c4 = *(const u32x4*)(h + 4 * lane);
    const uint32_t lsum = c4[0] + c4[1] + c4[2] + c4[3];
    uint32_t suf = lsum;  // inclusive suffix sum over lanes >= this one
#pragma unroll
    for (int d = 1; d < kWave; d <<= 1) {
      const uint32_t o = __shfl_down(suf, d, kWave);
      suf += lane + d < kWave ? o : 0u;
    }
    const uint32_t need = kp - above;
    // the lane whose four digits hold the need-th key from the top
    const uint64_t hm = ballot(suf >= need && suf - lsum < need);
    const int hl = (int)__builtin_ctzll(hm | (1ull << 63));
    uint32_t dsel = 0, abv = 0, neq = 0;
    {
      uint32_t cum = suf - lsum;  // keys in the lanes above
      int dd = 3;
      for (; dd > 0; --dd) {
        if (cum + c4[dd] >= need) break;
        cum += c4[dd];
      }
      dsel = 4u * (uint32_t)lane + (uint32_t)dd;
      abv = cum;
      neq = c4[dd];
    }
    dsel = sgpr(__builtin_amdgcn_readlane(dsel, hl));
    above += sgpr(__builtin_amdgcn_readlane(abv, hl));
    n_eq = sgpr(__builtin_amdgcn_readlane(neq, hl));
    pre = (rd == 0 ? 0u : pre << 8) | dsel;
    sh_prev = sh;
  }
  const uint32_t t = lo + pre;             // the kp-th largest gathered key
  const uint32_t need = kp - above;        // keys equal to t that are kept, >= 1
  uint32_t i_last = kAllTies;
  if (n_eq != need) {
    // the need-th smallest index among keys equal to t: their bits in the
    // cleared bitmap of the block's indices, each thread's 256 bits
    // counted, a workgroup prefix
#pragma unroll
    for (int r = 0; r < NR; ++r)
      if (y[r] == pre) {
        const uint32_t ix = myidx[lane + kWave * r];
        atomicOr(&bits[ix >> 5], 1u << (ix & 31u));
      }
    lds_sync();
    constexpr int WPT = kMaxBlock / 32 / kThrThreads;  // words per thread: 8
    uint32_t wv[WPT], c = 0;
#pragma unroll
    for (int q = 0; q < WPT; ++q) {
      const uint32_t at = (uint32_t)tid * WPT + q;
      wv[q] = at < nw32 ? bits[at] : 0u;
      c += (uint32_t)__builtin_popcount(wv[q]);
    }
    // exclusive prefix of c (< 2^9) over the workgroup's threads
    uint32_t in_wave = 0, wave_total = 0;
#pragma unroll
    for (int b2 = 0; b2 < 9; ++b2) {
      const uint64_t m = ballot((c >> b2) & 1u);
      in_wave += lanes_below(m) << b2;
      wave_total += popc(m) << b2;
    }
    if (lane == 0) cnt[wave] = wave_total;
    lds_sync();
    uint32_t before = in_wave;
#pragma unroll
    for (int w = 0; w < kThrWaves; ++w) before += w < wave ? cnt[w] : 0u;
    if (before < need && before + c >= need) {
      uint32_t r2 = need - before;  // the r2-th set bit of this thread's words
      uint32_t found = 0;
#pragma unroll
      for (int q = 0; q < WPT; ++q) {
        const uint32_t pc = (uint32_t)__builtin_popcount(wv[q]);
        if (found == 0 && r2 <= pc) {
          uint32_t x = wv[q];
          for (uint32_t z = 1; z < r2; ++z) x &= x - 1u;  // drop the lower set bits
          found = ((uint32_t)tid * WPT + q) * 32u + (uint32_t)__builtin_ctz(x) + 1u;
        }
        if (found == 0) r2 -= pc;
      }
      misc[0] = found - 1u;
    }
    lds_sync();
    i_last = sgpr(misc[0]);
  }
  // kept gathered keys per sub-block, then the row positions
#pragma unroll
  for (int r = 0; r < NR; ++r) {
    const uint32_t q = (uint32_t)(lane + kWave * r);
    if (q < mine) {
      const uint32_t ix = myidx[q];
      const bool kept = y[r] > pre || (y[r] == pre && (i_last == kAllTies || ix <= i_last));
      if (kept) atomicAdd(&kept_sb[ix >> 12], 1u);
    }
  }
  lds_sync();
  if (tid < 16) {
    uint32_t off = 0;
    for (int w = 0; w < tid; ++w) off += hi_sb[w] + kept_sb[w];
    __builtin_amdgcn_raw_buffer_store_b32(off < (uint32_t)kq ? off : (uint32_t)kq, rrec, 16 + 4 * tid, 0, 0);
  } else if (tid == 16) {
    __builtin_amdgcn_raw_buffer_store_b128(u32x4{1u, t, i_last, 0u}, rrec, 0, 0, 0);
  }
}

// -------------------------------------------------------- apply kernel
// One wave per 4096-element sub-block w of a block the threshold kernel
// settled: lane l owns the sub-block's elements [64l, 64l + 64), loaded and
// decoded as in the one-wave select; kept are |a| > T and |a| == T up to
// i_last.  The kept elements go to the row from the record's position of
// the sub-block, in element order, and the segment table gets the row
// position of each of its four 1024-element quarters' first entry.
template <bool LB, bool GBF16, bool VF32, int EFM>
__global__ void __launch_bounds__(kWave) __attribute__((amdgpu_waves_per_eu(4)))
apply_kernel(StepParams p, int64_t first, int64_t count, int32_t nsb) {
  constexpr int EPL = 64, NV = EPL / 8, CAP = kWave * EPL;
  using E = Entry<VF32>;
  extern __shared__ __align__(16) uint32_t smem[];
  const int lane = thread_id();
  const int64_t w = xcd_block(block_id(), count * nsb);
  const int64_t gb = first + w / nsb;
  const int sb = (int)(w % nsb);
  const Rsrc rrec = make_rsrc(p.thr + (uint64_t)gb * kThrRecordBytes, kThrRecordBytes);
  const u32x4 head = __builtin_amdgcn_raw_buffer_load_b128(rrec, 0, 0, 0);
  const uint32_t off0 = sgpr(__builtin_amdgcn_raw_buffer_load_b32(rrec, 16 + 4 * sb, 0, 0));
  if (sgpr(head[0]) == 0u) return;  // the multi-wave select takes this block
  const uint32_t T = sgpr(head[1]), i_last = sgpr(head[2]);
  const int bl = p.bucket_log2;
  const uint32_t e_sb = (uint32_t)sb * CAP;
  const uint32_t eb = (uint32_t)lane * EPL;

  const uint32_t sub_ef = (EFM & kEf8) ? (uint32_t)CAP : (uint32_t)CAP / 2;
  const uint32_t ef_bytes = (EFM & kEf8) ? (uint32_t)p.block : (uint32_t)(p.block >> 1);
  const uint32_t nbk = (uint32_t)(p.block >> bl), sub_bk = (uint32_t)(CAP >> bl);
  const Rsrc re = make_rsrc(p.state + p.ef_plane + (uint64_t)gb * ef_bytes + (uint64_t)sb * sub_ef, sub_ef);
  const Rsrc rs = make_rsrc(p.state + p.stats_plane + ((uint64_t)gb * nbk + (uint64_t)sb * sub_bk) * 8, sub_bk * 8);
  constexpr bool kCoal = GBF16;
  LaneIn<EPL, LB, GBF16, EFM> in;
  CoalescedIn cx;
  if constexpr (kCoal) {
#pragma unroll
    for (int v = 0; v < (LB ? 1 : NV); ++v)
      in.st[v] = __builtin_amdgcn_raw_buffer_load_b64(rs, ((eb + 8 * v) >> bl) * 8, 0, kStream);
    coalesced_load_codes<EFM>(cx, re, lane);
  } else {
    lane_load_state(in, re, rs, eb, bl, true);
  }
  const Block b = locate(p, gb);
  const int s_blk = b.s, kq = b.kq;
  const int nq = p.block / kQuarter;  // segment table entries per row
  constexpr uint32_t EB = VF32 ? 8u : 4u;
  const uint32_t table = (uint32_t)p.window * p.k_full * EB;
  const Rsrc rwin = make_rsrc(p.state + p.win_plane + (uint64_t)gb * p.win_stride, (uint32_t)p.win_stride);
  auto table_store = [&](int quarter, uint32_t pos) {
    __builtin_amdgcn_raw_buffer_store_b32(pos < (uint32_t)kq ? pos : (uint32_t)kq, rwin,
                                          table + ((uint32_t)p.new_slot * nq + quarter) * 4, 0, 0);
  };
  const int s = s_blk - (int)e_sb;  // this sub-block's elements (may be <= 0)
  if (s <= 0) {
    if (lane < 4) table_store(4 * sb + lane, off0);
    return;
  }
  const bool full = s >= CAP;
  const int ss = full ? CAP : s;
  const Rsrc rg = make_rsrc((const uint8_t*)b.desc.grad + (b.e0 + e_sb) * (GBF16 ? 2 : 4), vec_bytes<GBF16>(ss));
  if constexpr (kCoal) {
    coalesced_load_grad(cx, rg, lane);
    coalesced_exchange(cx, in, smem, lane);
  } else {
    lane_load_grad(in, rg, eb);
  }
  float a[NV][8];
  const int rem = ss - (int)eb;
  lane_decode(in, a, rem, full);

  // kept elements: a set per lane, positioned in element order, written to
  // the row
  const bool notie = i_last == kAllTies;
  // i_last relative to this lane's first element (negative: no tie kept here)
  const int last_here = notie ? CAP : (int)i_last - (int)e_sb - (int)eb;
  const float tf = opaque_f(__uint_as_float(T));
  // kept: |a| >= T when every key equal to T is kept (the common case), else
  // |a| > T and |a| == T up to i_last
  auto kept = [&](auto notie_tag, float ab, int i) {
    if constexpr (decltype(notie_tag)::value) return ab >= tf;
    else return (ab > tf) | ((ab == tf) & (i <= last_here));
  };
  // the lane's kept set: element i at bit 31 - (i mod 32) of word i / 32, so
  // that the leading zeros of a word lead to its next kept element.  With
  // bf16 entries the lane's values go to LDS first (element i at halfword i
  // of the lane's 128 bytes; the exchange is over), and the kept elements
  // are zeroed for the quantization as they are marked.
  if constexpr (!VF32) {
#pragma unroll
    for (int v = 0; v < NV; ++v) {
      u32x4 x;
#pragma unroll
      for (int h = 0; h < 4; ++h) x[h] = pack_bf16x2(a[v][2 * h], a[v][2 * h + 1]);
      *(u32x4*)(smem + 32 * lane + 4 * v) = x;
    }
    __builtin_amdgcn_sched_barrier(0);  // (the packed words die here)
  }
  // The mask of lanes whose element i is a tie kept by index: lane l holds
  // element 64 l + i of the sub-block, kept when 64 l + i <= R (R: i_last in
  // the sub-block), i.e. the lanes [0, floor((R - i) / 64)], which is
  // [0, q] for i <= R mod 64 and [0, q - 1] above (q = floor(R / 64)).
  // Without ties past the threshold every tie is kept: R beyond the block.
  const int R = notie ? 2 * CAP : (int)i_last - (int)e_sb;
  const int q = R >> 6, r_mod = R & 63;
  auto lanes_upto = [](int last) -> uint64_t {
    return last < 0 ? 0ull : last >= kWave - 1 ? ~0ull : (2ull << last) - 1ull;
  };
  const uint64_t ties_hi = lanes_upto(q), ties_lo = lanes_upto(q - 1);
  uint32_t km[2] = {0u, 0u};
#pragma unroll
  for (int v = 0; v < NV; ++v)
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      uint32_t& w = km[v / (NV / 2)];
      const float ab = __builtin_fabsf(a[v][e]);
      // (the set's mask combined from the compares' own masks)
      const uint64_t m = ballot(ab > tf) | (ballot(ab == tf) & (8 * v + e <= r_mod ? ties_hi : ties_lo));
      if constexpr (VF32) w = shift_in_mask(w, m);
      else w = shift_in_mask_zero(w, m, a[v][e]);
    }
  const uint32_t sel_l = (uint32_t)__builtin_popcount(km[0]) + (uint32_t)__builtin_popcount(km[1]);
  uint32_t pre = 0, n_sb = 0;  // kept before this lane; in the sub-block
#pragma unroll
  for (int b2 = 0; b2 < 7; ++b2) {
    const uint64_t m = ballot((sel_l >> b2) & 1u);
    pre += lanes_below(m) << b2;
    n_sb += popc(m) << b2;
  }
  n_sb = sgpr(n_sb);
  if ((lane & 15) == 0 && 4 * sb + (lane >> 4) < nq) table_store(4 * sb + (lane >> 4), off0 + pre);
  // the sub-block's entries that enter the row, [off0, off0 + n_row), are
  // staged in LDS and leave as consecutive words; past kApplyStageWords
  // each is stored where it is found
  constexpr uint32_t EW = VF32 ? 2u : 1u;
  const uint32_t room = off0 < (uint32_t)kq ? (uint32_t)kq - off0 : 0u;
  const uint32_t n_row = n_sb < room ? n_sb : room;
  const bool staged = n_row * EW <= kApplyStageWords;
  const Rsrc rw = window_rsrc<VF32 ? 2 : 1>(p, gb, kq);
  const uint32_t row0 = (uint32_t)p.new_slot * kq + off0;
  // (every kept entry fits the row unless the threshold pass kept more than
  // k_q, which it does not; the bound check stays for that case)
  uint32_t* const stage = smem + (VF32 ? 0u : kApplyValWords);
  if constexpr (!VF32) {
    // bf16 entries: each lane walks its kept set, reading each value back
    // from LDS by its element number
    wave_sync();
    const uint16_t* const vals = (const uint16_t*)smem + 64 * lane;
    const uint32_t idx0 = e_sb + eb;
    auto walk = [&](auto staged_tag) {
      constexpr bool STAGED = decltype(staged_tag)::value;
      uint32_t r = pre;
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        uint32_t m = km[h];
        while (m != 0u) {
          const uint32_t e = (uint32_t)__builtin_clz(m);
          m ^= 0x80000000u >> e;
          const uint32_t i = 32u * (uint32_t)h + e;
          const uint32_t x = (idx0 + i) | ((uint32_t)vals[i] << 16);  // the entry of element i
          if (r < n_row) {
            if constexpr (STAGED) stage[r] = x;
            else E::store(rw, row0 + r, x);
          }
          ++r;
        }
      }
    };
    if (staged)
      walk(BoolTag<true>{});
    else
      walk(BoolTag<false>{});
  } else {
    // binary32 entries: each kept element written from its register
    auto write_row = [&](auto notie_tag, auto staged_tag) {
      constexpr bool STAGED = decltype(staged_tag)::value;
      uint32_t r = pre;
#pragma unroll
      for (int v = 0; v < NV; ++v) {
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          if (kept(notie_tag, __builtin_fabsf(a[v][e]), 8 * v + e)) {
            if (r < n_row) {
              const typename E::T x = E::make(e_sb + eb + 8 * v + e, a[v][e]);
              if constexpr (STAGED) *(u32x2*)(stage + 2 * r) = x;
              else E::store(rw, row0 + r, x);
            }
            ++r;
          }
        }
        __builtin_amdgcn_sched_barrier(0);  // one vector's stores at a time
      }
    };
    if (sel_l) {
      if (notie && staged)
        write_row(BoolTag<true>{}, BoolTag<true>{});
      else if (staged)
        write_row(BoolTag<false>{}, BoolTag<true>{});
      else
        write_row(BoolTag<false>{}, BoolTag<false>{});
    }
  }
  if (staged) {
    wave_sync();
    for (uint32_t q = (uint32_t)lane; q < n_row * EW; q += kWave)
      __builtin_amdgcn_raw_buffer_store_b32(stage[q], rw, (row0 * EW + q) * 4, 0, kStream);
  }
  // ---------------------------------------------- e = Q(a with a[I] = 0)
  lane_quantize_store<EPL, LB, EFM, !VF32>(a, T, notie, (uint32_t)((int)i_last - (int)e_sb), eb, ss, rem, full, bl,
                                           true, re, rs,
                                           EfStream{b.e0 + (int64_t)e_sb, b.j, (uint32_t)p.t, p.seed_lo, p.seed_hi},
                                           kCoal ? smem : nullptr);
}

template <bool GB, bool VF, int EFM>
hipError_t launch_select_split(const StepParams& p, int64_t first, int64_t count, hipStream_t stream) {
  if (count <= 0) return hipSuccess;
  hipLaunchKernelGGL((threshold_kernel<GB, EFM>), dim3((uint32_t)count), dim3(kThrThreads), ThrLds::kWords * 4,
                     stream, p, first, count);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int32_t nsb = p.block / kSubBlock;
  const size_t lds = apply_lds_words() * 4;
  if ((1 << p.bucket_log2) >= 64)
    hipLaunchKernelGGL((apply_kernel<true, GB, VF, EFM>), dim3((uint32_t)(count * nsb)), dim3(kWave), lds, stream, p,
                       first, count, nsb);
  else
    hipLaunchKernelGGL((apply_kernel<false, GB, VF, EFM>), dim3((uint32_t)(count * nsb)), dim3(kWave), lds, stream, p,
                       first, count, nsb);
  return hipGetLastError();
}

}  // namespace
}  // namespace microadam
