/*
 * MicroAdam CPU oracle.  TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, single-threaded statement of one MicroAdam optimizer step
 * over one parameter tensor, written from the paper "MicroAdam: Accurate
 * Adaptive Optimization with Low Space Overhead and Provable Convergence"
 * (Modoranu et al., 2024):
 *   - Algorithm 1 (MicroAdam with quantized error feedback),
 *   - Algorithm 2 (the AdamStats, Q and Q^-1 procedures),
 *   - Section 3.1 (Top-K applied per block of B_d elements with
 *     block-relative indices; per-bucket quantization metadata delta/Delta;
 *     the 4-bit error feedback stored two codes per byte),
 *   - Algorithm 4 (decoupled weight decay (1 - eta*lambda) * theta),
 *   - Lemma 1 (Section 4: the randomized-rounding quantizer of the error
 *     feedback, floor((x - delta)/u + xi) with xi ~ U[0, 1)), as an option
 *     beside the round-to-nearest Q of Algorithm 2; b = 4 or 8 bits.
 *
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg
 * load this library.  It shares no code, header or table with the HIP path.
 *
 * Precision.
 *   Everything that decides an integer -- the error-feedback decode, the
 *   accumulator, the Top-K choice, the bucket min/max, the 4-bit codes and
 *   the bf16 window value -- is IEEE binary32 with exactly one rounding per
 *   written operation (this file must be built with -ffp-contract=off and
 *   without fast-math).  The rounding mode is round-half-to-even throughout.
 *   The window-to-moment rebuild and the parameter update are binary64 and
 *   are rounded once, to the parameter's storage type, at the end.
 *
 * Readings of the paper taken here (each is listed with its reason in the
 * design notes of the repository):
 *   - k per block is ceil(density * s) for a block of s elements
 *     (at least 1, at most s);
 *   - Top-K ranks by |a|; ties go to the lower index; a row keeps the chosen
 *     entries in ascending index order with their signed values;
 *   - Q rounds half-to-even; a bucket whose max equals its min encodes every
 *     element as 0, and Q^-1 of any code in such a bucket is its min;
 *   - the randomized Q draws xi for element i of tensor j at step t from
 *     Philox4x32-10 (Salmon et al., "Parallel Random Numbers: As Easy as
 *     1, 2, 3", SC 2011): key = the 64-bit seed, counter = (i/4 low word,
 *     i/4 high word, j, t); word i mod 4 of the output, w, gives
 *     xi = (w >> 8) * 2^-24; the code is floor(y + xi) taken exactly (not
 *     after rounding the sum) for y = fl(fl(x - delta)/u), clamped to
 *     [0, 2^b - 1];
 *   - the window row written at step s is row (s-1) mod m; in AdamStats it
 *     carries the weight beta^(t-s), so the newest row has exponent 0 and the
 *     oldest m-1 (Section 3, "Dynamic Statistics");
 *   - the bias correction uses the global step: (1-beta)/(1-beta^t);
 *   - epsilon is added outside the square root, as in Algorithm 1;
 *   - weight decay is decoupled and dense, as in Algorithm 4;
 *   - a bucket min or max equal to -0 is stored as +0.
 *
 * Data layout (the oracle's own):
 *   theta[n], grad[n]     binary32 values (bf16 values held exactly)
 *   ef[(n+1)/2]           4-bit codes, element 2j in the low nibble
 *   ef[n]                 (b = 8) one code per byte
 *   delta[nb], Delta[nb]  bucket min / max, nb = ceil(n / B_q)
 *   win_idx[m*K]          window indices, row-major (m rows of K entries);
 *   win_val[m*K]          window values (bf16-rounded when value_bf16);
 *                         K = sum over blocks of k_q and block q's entries
 *                         occupy [q*k_full, q*k_full + k_q) of every row.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

typedef struct {
  int64_t n;          /* elements in the tensor                          */
  int32_t block;      /* B_d: Top-K block size                           */
  int32_t bucket;     /* B_q: quantization bucket size (divides B_d, or  */
                      /* any size when a step covers the whole tensor)   */
  int32_t window;     /* m: rows in the sliding window                   */
  int32_t value_bf16; /* 1: window values stored as bf16, 0: binary32    */
  int32_t param_bf16; /* 1: parameters stored as bf16, 0: binary32       */
  int32_t ef_bits;    /* b: 4 or 8                                       */
  double density;     /* k/d in (0, 1]                                   */
  double beta1, beta2, eps, weight_decay;
  int32_t rounding;   /* 0: nearest (Algorithm 2), 1: randomized (Lemma 1) */
  int32_t tensor;     /* j: the tensor's number, part of the random counter */
  uint64_t seed;      /* key of the random stream                        */
  int64_t offset;     /* number of this state's element 0 in its tensor  */
                      /* (part of the random counter; 0 for a tensor)    */
} oracle_cfg;

/* ---------------------------------------------------------------------- */
/* Sizes                                                                   */
/* ---------------------------------------------------------------------- */

/* Entries kept by Top-K in a block of s elements: ceil(density * s), with
 * a 1e-9 guard so that products like 0.01 * 100 do not round up to 2. */
int64_t oracle_block_k(int64_t s, double density) {
  double x = ceil(density * (double)s - 1e-9);
  int64_t k = (int64_t)x;
  if (k < 1) k = 1;
  if (k > s) k = s;
  return k;
}

int64_t oracle_num_blocks(const oracle_cfg* c) {
  return (c->n + c->block - 1) / c->block;
}

int64_t oracle_num_buckets(const oracle_cfg* c) {
  return (c->n + c->bucket - 1) / c->bucket;
}

/* Width K of one window row: the sum of k_q over the tensor's blocks. */
int64_t oracle_row_width(const oracle_cfg* c) {
  int64_t nb = oracle_num_blocks(c), K = 0;
  for (int64_t q = 0; q < nb; ++q) {
    int64_t s = c->n - q * c->block;
    if (s > c->block) s = c->block;
    K += oracle_block_k(s, c->density);
  }
  return K;
}

static int64_t block_size(const oracle_cfg* c, int64_t q) {
  int64_t s = c->n - q * c->block;
  return s > c->block ? c->block : s;
}

static int64_t block_slot(const oracle_cfg* c, int64_t q) {
  return q * oracle_block_k(c->block, c->density);
}

/* ---------------------------------------------------------------------- */
/* bf16 rounding: nearest bf16 value of x, ties to even (8 significant     */
/* bits, the binary32 exponent range, bf16 subnormals spaced 2^-133).      */
/* ---------------------------------------------------------------------- */
static float round_to_bf16(double x) {
  if (x == 0.0 || !isfinite(x)) return (float)x;
  int e;
  (void)frexp(x, &e);         /* |x| in [2^(e-1), 2^e) */
  int q = e - 8;              /* bf16 spacing in that binade */
  if (q < -133) q = -133;     /* subnormal spacing */
  double r = nearbyint(ldexp(x, -q)); /* exact scaling, then RNE */
  return (float)ldexp(r, q);  /* exact; 2^128 and above become inf */
}

/* ---------------------------------------------------------------------- */
/* Q and Q^-1 (Algorithm 2; Lemma 1), binary32, L = 2^b - 1 levels         */
/* ---------------------------------------------------------------------- */

/* Q^-1: x = x_Q * u + delta with u = (Delta - delta) / (2^b - 1). */
static float dequantize(unsigned code, float lo, float hi, float levels) {
  float u = (hi - lo) / levels;
  float scaled = (float)code * u;
  return scaled + lo;
}

/* Q: x_Q = round((x - delta) / u), rounding half to even, kept in [0, L];
 * a bucket with u == 0 encodes 0. */
static unsigned quantize(float x, float lo, float hi, float levels) {
  float u = (hi - lo) / levels;
  if (u == 0.0f) return 0u;
  float y = (x - lo) / u;
  float r = nearbyintf(y);
  if (r < 0.0f) r = 0.0f;
  if (r > levels) r = levels;
  return (unsigned)r;
}

/* Randomized Q (Lemma 1): x_Q = floor((x - delta) / u + xi), kept in
 * [0, L]; a bucket with u == 0 encodes 0.  xi = w * 2^-24 for a 24-bit
 * integer w, and the floor of the exact sum y + xi is floor(y) + 1 exactly
 * when w + floor(2^24 * frac(y)) >= 2^24 (frac(y) and its scaling are exact
 * in binary32); rounding the sum first would move y's just below an integer
 * up with a probability of up to one ulp. */
static unsigned quantize_randomized(float x, float lo, float hi, float levels, uint32_t w24) {
  float u = (hi - lo) / levels;
  if (u == 0.0f) return 0u;
  float y = (x - lo) / u;
  float fy = floorf(y);
  float f = y - fy;
  uint32_t fr = (uint32_t)floorf(f * 16777216.0f);
  float r = fy + ((w24 + fr >= (1u << 24)) ? 1.0f : 0.0f);
  if (r < 0.0f) r = 0.0f;
  if (r > levels) r = levels;
  return (unsigned)r;
}

/* Philox4x32-10 (Salmon, Moraes, Dror and Shaw, SC 2011): ten rounds of
 * two 32x32 -> 64-bit products with the round keys, the key advancing by
 * the Weyl constants between rounds. */
static void philox4x32_10(const uint32_t ctr[4], uint32_t k0, uint32_t k1, uint32_t out[4]) {
  uint32_t x0 = ctr[0], x1 = ctr[1], x2 = ctr[2], x3 = ctr[3];
  for (int round = 0; round < 10; ++round) {
    if (round > 0) {
      k0 += 0x9E3779B9u;
      k1 += 0xBB67AE85u;
    }
    const uint64_t p0 = (uint64_t)0xD2511F53u * x0;
    const uint64_t p1 = (uint64_t)0xCD9E8D57u * x2;
    const uint32_t y0 = (uint32_t)(p1 >> 32) ^ x1 ^ k0;
    const uint32_t y1 = (uint32_t)p1;
    const uint32_t y2 = (uint32_t)(p0 >> 32) ^ x3 ^ k1;
    const uint32_t y3 = (uint32_t)p0;
    x0 = y0; x1 = y1; x2 = y2; x3 = y3;
  }
  out[0] = x0; out[1] = x1; out[2] = x2; out[3] = x3;
}

/* The 24-bit integer w of xi = w * 2^-24 for element i of tensor j at step
 * t: xi is uniform on [0, 1) in steps of 2^-24. */
static uint32_t uniform_w24(uint64_t seed, int32_t j, int64_t t, int64_t i) {
  const uint64_t quad = (uint64_t)i >> 2;
  const uint32_t ctr[4] = {(uint32_t)quad, (uint32_t)(quad >> 32), (uint32_t)j, (uint32_t)t};
  uint32_t out[4];
  philox4x32_10(ctr, (uint32_t)seed, (uint32_t)(seed >> 32), out);
  return out[i & 3] >> 8;
}

static unsigned get_code(const uint8_t* ef, int64_t i, int bits) {
  if (bits == 8) return ef[i];
  uint8_t byte = ef[i >> 1];
  return (i & 1) ? (unsigned)(byte >> 4) : (unsigned)(byte & 0x0F);
}

static void put_code(uint8_t* ef, int64_t i, unsigned code, int bits) {
  if (bits == 8) {
    ef[i] = (uint8_t)code;
    return;
  }
  uint8_t byte = ef[i >> 1];
  if (i & 1) byte = (uint8_t)((byte & 0x0F) | (code << 4));
  else       byte = (uint8_t)((byte & 0xF0) | code);
  ef[i >> 1] = byte;
}

/* ---------------------------------------------------------------------- */
/* Top-K of |a| over one block (Section 3.1): ties to the lower index.      */
/* ---------------------------------------------------------------------- */
static const float* g_sort_vals; /* single-threaded: qsort has no context */

static int by_magnitude_then_index(const void* pa, const void* pb) {
  int32_t i = *(const int32_t*)pa, j = *(const int32_t*)pb;
  float ai = fabsf(g_sort_vals[i]), aj = fabsf(g_sort_vals[j]);
  if (ai > aj) return -1;
  if (ai < aj) return 1;
  return (i < j) ? -1 : (i > j);
}

static int ascending(const void* pa, const void* pb) {
  int32_t i = *(const int32_t*)pa, j = *(const int32_t*)pb;
  return (i > j) - (i < j);
}

/* Writes the k largest-|a| positions of a[0..s), in ascending order. */
static void topk_block(const float* a, int64_t s, int64_t k, int32_t* out) {
  int32_t* order = (int32_t*)malloc(sizeof(int32_t) * (size_t)s);
  for (int64_t i = 0; i < s; ++i) order[i] = (int32_t)i;
  g_sort_vals = a;
  qsort(order, (size_t)s, sizeof(int32_t), by_magnitude_then_index);
  memcpy(out, order, sizeof(int32_t) * (size_t)k);
  qsort(out, (size_t)k, sizeof(int32_t), ascending);
  free(order);
}

/* ---------------------------------------------------------------------- */
/* AdamStats (Algorithm 2) over blocks [q0, q1): dense binary64 output for */
/* elements [q0*B_d, min(n, q1*B_d)).                                      */
/* ---------------------------------------------------------------------- */
static void adam_stats(const oracle_cfg* c, int64_t t, double beta, int squared,
                       const uint16_t* win_idx, const float* win_val,
                       int64_t q0, int64_t q1, double* out) {
  const int64_t m = c->window, K = oracle_row_width(c);
  const int64_t base = q0 * c->block;
  int64_t end = q1 * c->block;
  if (end > c->n) end = c->n;
  for (int64_t i = base; i < end; ++i) out[i - base] = 0.0;   /* z <- 0 */
  int64_t first = t - m + 1;
  if (first < 1) first = 1;
  for (int64_t s = first; s <= t; ++s) {       /* oldest row first */
    const int64_t row = (s - 1) % m;
    const double w = pow(beta, (double)(t - s)); /* beta^r, r = t - s */
    for (int64_t q = q0; q < q1; ++q) {
      const int64_t k = oracle_block_k(block_size(c, q), c->density);
      const int64_t slot = row * K + block_slot(c, q);
      for (int64_t j = 0; j < k; ++j) {
        const double v = (double)win_val[slot + j];
        const int64_t i = q * c->block + (int64_t)win_idx[slot + j];
        out[i - base] += w * (squared ? v * v : v);
      }
    }
  }
  const double scale = (1.0 - beta) / (1.0 - pow(beta, (double)t));
  for (int64_t i = base; i < end; ++i) out[i - base] *= scale;
}

/* Dense m-hat and v-hat of the current window for blocks [q0, q1). */
void oracle_moments(const oracle_cfg* c, int64_t t, const uint16_t* win_idx,
                    const float* win_val, int64_t q0, int64_t q1,
                    double* mhat, double* vhat) {
  adam_stats(c, t, c->beta1, 0, win_idx, win_val, q0, q1, mhat);
  adam_stats(c, t, c->beta2, 1, win_idx, win_val, q0, q1, vhat);
}

/* ---------------------------------------------------------------------- */
/* One MicroAdam step (Algorithm 1) at step t >= 1 over blocks [q0, q1).   */
/* Blocks are independent: every quantity a block reads or writes belongs  */
/* to that block, so a sub-range gives exactly the full run's values there. */
/* ---------------------------------------------------------------------- */
int oracle_step(const oracle_cfg* c, int64_t t, double lr, float* theta,
                const float* grad, uint8_t* ef, float* delta, float* Delta,
                uint16_t* win_idx, float* win_val, int64_t q0, int64_t q1) {
  if (t < 1 || c->window < 1 || c->block < 1 || c->bucket < 1 ||
      (c->ef_bits != 4 && c->ef_bits != 8) || (c->rounding != 0 && c->rounding != 1))
    return -1;
  const int64_t nblk = oracle_num_blocks(c);
  if (q1 > nblk) q1 = nblk;
  if (q0 < 0 || q0 >= q1) return 0;
  /* a bucket that does not lie inside one block needs the whole tensor */
  if (c->block % c->bucket != 0 && (q0 != 0 || q1 != nblk)) return -1;
  const float levels = (float)((1 << c->ef_bits) - 1);
  const int64_t lo = q0 * c->block;
  int64_t hi = q1 * c->block;
  if (hi > c->n) hi = c->n;
  const int64_t len = hi - lo, K = oracle_row_width(c), m = c->window;
  const int64_t row = (t - 1) % m;             /* the circular pointer i */

  float* a = (float*)malloc(sizeof(float) * (size_t)len);
  int32_t* chosen = (int32_t*)malloc(sizeof(int32_t) * (size_t)c->block);

  /* Accumulator: a = g + Q^-1(e, delta, Delta). */
  for (int64_t i = lo; i < hi; ++i) {
    const int64_t b = i / c->bucket;
    a[i - lo] = grad[i] + dequantize(get_code(ef, i, c->ef_bits), delta[b], Delta[b], levels);
  }

  for (int64_t q = q0; q < q1; ++q) {
    const int64_t s = block_size(c, q), k = oracle_block_k(s, c->density);
    float* ab = a + (q * c->block - lo);
    /* I, V = T_k(|a|) per block, written to window row i in index order. */
    topk_block(ab, s, k, chosen);
    const int64_t slot = row * K + block_slot(c, q);
    for (int64_t j = 0; j < k; ++j) {
      const float v = ab[chosen[j]];
      win_idx[slot + j] = (uint16_t)chosen[j];
      win_val[slot + j] = c->value_bf16 ? round_to_bf16((double)v) : v;
    }
    /* a[I] = 0: the kept entries leave the error feedback. */
    for (int64_t j = 0; j < k; ++j) ab[chosen[j]] = 0.0f;
  }

  /* delta, Delta = min(a), max(a) per bucket; e = Q(a, delta, Delta). */
  for (int64_t b0 = lo; b0 < hi; b0 += c->bucket) {
    int64_t b1 = b0 + c->bucket;
    if (b1 > hi) b1 = hi;
    float mn = a[b0 - lo], mx = a[b0 - lo];
    for (int64_t i = b0; i < b1; ++i) {
      if (a[i - lo] < mn) mn = a[i - lo];
      if (a[i - lo] > mx) mx = a[i - lo];
    }
    if (mn == 0.0f) mn = 0.0f; /* -0 stored as +0 */
    if (mx == 0.0f) mx = 0.0f;
    const int64_t b = b0 / c->bucket;
    delta[b] = mn;
    Delta[b] = mx;
    for (int64_t i = b0; i < b1; ++i) {
      const unsigned code = c->rounding
          ? quantize_randomized(a[i - lo], mn, mx, levels, uniform_w24(c->seed, c->tensor, t, c->offset + i))
          : quantize(a[i - lo], mn, mx, levels);
      put_code(ef, i, code, c->ef_bits);
    }
  }

  /* m-hat, v-hat = AdamStats over the window (binary64), then the update
   * theta <- (1 - eta*lambda) theta - eta * m / (eps + sqrt(v)). */
  double* mh = (double*)malloc(sizeof(double) * (size_t)len);
  double* vh = (double*)malloc(sizeof(double) * (size_t)len);
  oracle_moments(c, t, win_idx, win_val, q0, q1, mh, vh);
  const double decay = 1.0 - lr * c->weight_decay;
  for (int64_t i = lo; i < hi; ++i) {
    const double upd = mh[i - lo] / (c->eps + sqrt(vh[i - lo]));
    const double nt = (double)theta[i] * decay - lr * upd;
    theta[i] = c->param_bf16 ? round_to_bf16(nt) : (float)nt;
  }

  free(mh);
  free(vh);
  free(chosen);
  free(a);
  return 0;
}

/* Exposed for the tests: binary32 -> bf16 rounding and the codec. */
float oracle_round_bf16(double x) { return round_to_bf16(x); }
float oracle_dequantize(unsigned code, float lo, float hi, int bits) {
  return dequantize(code, lo, hi, (float)((1 << bits) - 1));
}
unsigned oracle_quantize(float x, float lo, float hi, int bits) {
  return quantize(x, lo, hi, (float)((1 << bits) - 1));
}
/* xi must lie on the 2^-24 grid of [0, 1). */
unsigned oracle_quantize_randomized(float x, float lo, float hi, int bits, float xi) {
  return quantize_randomized(x, lo, hi, (float)((1 << bits) - 1), (uint32_t)(xi * 16777216.0f));
}
void oracle_philox4x32_10(const uint32_t ctr[4], uint32_t k0, uint32_t k1, uint32_t out[4]) {
  philox4x32_10(ctr, k0, k1, out);
}
float oracle_uniform_xi(uint64_t seed, int32_t j, int64_t t, int64_t i) {
  return (float)uniform_w24(seed, j, t, i) * 0x1p-24f;
}
