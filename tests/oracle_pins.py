"""Pins for the CPU oracle: checks against what the MicroAdam paper and plain
mathematics fix, never against the oracle's own formulas.

Each ``check_*`` function takes an ``oracle.Oracle`` and raises
``AssertionError`` on a mismatch.  ``test_oracle_pins.py`` runs them on the
real oracle; ``test_oracle_mutants.py`` runs them on deliberately broken
builds of the oracle source and requires every break to be caught.

What pins what:
  - Top-K: brute-force full sort with lower-index-wins ties (Section 3.1);
    the Top-K contraction bound of Assumption 1 per block.
  - Q / Q^-1 (Algorithm 2): half-step error bound, min -> code 0 decoding
    exactly, max -> code 15, all-equal bucket -> 0, half-to-even on exact
    half steps, monotone codes.
  - Error feedback (Algorithm 1): bucket min/max of the residual recomputed
    by numpy; the reconstruction decode(e_{t+1}) + V ~= a_t.
  - AdamStats: with density 1 the window moments are Adam's bias-corrected
    EMA (t <= m, Adam recurrence) or its m-term truncation (t > m, a sliding
    recurrence); m = 1 closed form; a spike per step pins beta^(t-s) and which
    rows are live (Section 3, "Dynamic Statistics").
  - Update: the t = 1 closed form theta - eta*V/(eps+|V|) on the kept
    entries; untouched entries bit-identical for lambda = 0; decoupled decay
    (1 - eta*lambda)*theta elsewhere (Algorithm 4).
  - bf16 rounding: torch's CPU float32 -> bfloat16 conversion (RNE), and a
    binary64 double-rounding case.
  - bf16 parameters (Algorithm 1's update stored in bf16): the t = 1 closed
    form rounded once from binary64 (round to odd into binary32, then torch's
    RNE), including a value placed just off a bf16 midpoint so that a
    rounding through binary32 gives the other neighbour.
  - Buckets spanning Top-K blocks (Section 3.1 names buckets of 100K): the
    buckets are each tensor's element ranges [c*B_q, (c+1)*B_q), whatever the
    block size; after step 1 every bucket's (min, max) and codes are those of
    the residual over that range (numpy), and the reconstruction and Lemma 1
    norm bounds hold through several steps.
  - Randomized Q (Lemma 1): E[x_hat] = x, checked by averaging over xi on
    the midpoints of 256 equal cells of [0, 1) and, through whole steps, over
    300 seeds; every draw is one of the two grid points around x; the
    bucket's min and max are exact; the lemma's norm bound per bucket.
  - The random stream: the published known-answer vectors of Philox4x32-10
    (Salmon et al., SC 2011); xi on the 2^-24 grid of [0, 1), uniform
    (mean and a 16-bin chi-square), changing with seed, tensor and step.
  - 8-bit codes: the half-step bound with 255 levels, ties to even, max ->
    255, and the step's reconstruction bound.
"""
from __future__ import annotations

import math
from fractions import Fraction

import numpy as np
import torch

BETA1, BETA2, EPS = 0.9, 0.999, 1e-8


def _bf16(x) -> np.ndarray:
    """float32 -> bf16 (round-half-to-even) by torch's CPU conversion."""
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t.to(torch.bfloat16).to(torch.float32).numpy()


def _bf16_from_f64(x) -> np.ndarray:
    """binary64 -> bf16 with one rounding (half to even): round to odd into
    binary32 (truncate toward zero, then set the last bit when inexact), then
    torch's binary32 -> bf16 conversion.  Rounding to odd into a format with
    at least two more bits than the target makes the second rounding the
    correct one (Boldo and Melquiond, IEEE Trans. Computers 57(4), 2008).
    (torch's own float64 -> bfloat16 goes through binary32 with two roundings
    to nearest, which is what the pins must tell apart.)"""
    x = np.asarray(x, np.float64)
    f = x.astype(np.float32)
    over = np.abs(f.astype(np.float64)) > np.abs(x)
    f = np.where(over, np.nextafter(f, np.float32(0)), f).astype(np.float32)
    inexact = (f.astype(np.float64) != x).astype(np.uint32)
    return _bf16((f.view(np.uint32) | inexact).view(np.float32))


def _brute_topk(x: np.ndarray, k: int) -> list[int]:
    """Positions of the k largest |x|, lower index first on ties, sorted."""
    order = sorted(range(len(x)), key=lambda i: (-abs(float(x[i])), i))
    return sorted(order[:k])


def _decode(codes, lo, hi, bucket, levels=15):
    """Q^-1 per element in binary32 (x_Q * u + delta, u = (Delta-delta)/L)."""
    b = np.arange(codes.size) // bucket
    u = ((hi[b] - lo[b]) / np.float32(levels)).astype(np.float32)
    return (codes.astype(np.float32) * u).astype(np.float32) + lo[b]


def _ulp(x) -> np.ndarray:
    return np.spacing(np.abs(np.asarray(x, np.float32))).astype(np.float64)


# ---------------------------------------------------------------------------
def check_round_bf16(o) -> None:
    rng = np.random.default_rng(11)
    xs = np.concatenate([
        rng.standard_normal(2000).astype(np.float32) * 10.0 ** rng.integers(-30, 30, 2000),
        # exact halfway cases with even and odd kept parts
        np.array([0x3F808000, 0x3F818000, 0xBF808000, 0x00008000, 0x00018000,
                  0x7F7F8000, 0x7F7FFFFF, 0x00000001, 0x80000001, 0x007FFFFF],
                 dtype=np.uint32).view(np.float32),
    ]).astype(np.float32)
    want = _bf16(xs)
    got = np.array([o.round_bf16(float(x)) for x in xs], np.float32)
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32)), "bf16 RNE"
    # binary64 input: 1 + 2^-8 + 2^-40 lies above the bf16 midpoint 1 + 2^-8,
    # so it rounds up; rounding through binary32 first would tie to 1.0.
    assert o.round_bf16(1.0 + 2.0 ** -8 + 2.0 ** -40) == 1.0 + 2.0 ** -7
    assert o.round_bf16(1.0 + 2.0 ** -8) == 1.0            # tie to even
    assert o.round_bf16(1.0 + 3 * 2.0 ** -8) == 1.0 + 2.0 ** -6


def check_quantizer(o) -> None:
    # half steps round to even: lo = 0, hi = 15 gives u = 1
    for x, want in [(0.5, 0), (1.5, 2), (2.5, 2), (3.5, 4), (14.5, 14), (0.49, 0),
                    (0.51, 1), (15.0, 15), (0.0, 0), (7.0, 7)]:
        assert o.quantize(x, 0.0, 15.0) == want, (x, want)
    assert o.quantize(3.0, 3.0, 3.0) == 0 and o.dequantize(0, 3.0, 3.0) == 3.0
    assert o.dequantize(9, -2.0, -2.0) == -2.0
    rng = np.random.default_rng(5)
    for _ in range(300):
        lo, hi = np.sort(rng.standard_normal(2).astype(np.float32) * np.float32(10.0 ** rng.integers(-6, 3)))
        lo, hi = float(lo), float(hi)
        u = (hi - lo) / 15.0
        assert o.quantize(lo, lo, hi) == 0 and o.dequantize(0, lo, hi) == lo
        if hi > lo:
            assert o.quantize(hi, lo, hi) == 15
        xs = np.sort(rng.uniform(lo, hi, 64).astype(np.float32))
        codes = [o.quantize(float(x), lo, hi) for x in xs]
        assert all(0 <= c <= 15 for c in codes)
        assert all(a <= b for a, b in zip(codes, codes[1:])), "codes not monotone"
        slack = 4 * float(_ulp(max(abs(lo), abs(hi))))
        for x, c in zip(xs, codes):
            assert abs(o.dequantize(c, lo, hi) - float(x)) <= u / 2 + slack, (x, lo, hi)


def check_quantizer_8bit(o) -> None:
    # 255 levels: lo = 0, hi = 255 gives u = 1, half steps round to even
    for x, want in [(0.5, 0), (1.5, 2), (2.5, 2), (100.5, 100), (254.5, 254), (255.0, 255),
                    (17.49, 17), (17.51, 18)]:
        assert o.quantize(x, 0.0, 255.0, 8) == want, (x, want)
    rng = np.random.default_rng(25)
    for _ in range(200):
        lo, hi = np.sort(rng.standard_normal(2).astype(np.float32) * np.float32(10.0 ** rng.integers(-6, 3)))
        lo, hi = float(lo), float(hi)
        u = (hi - lo) / 255.0
        assert o.quantize(lo, lo, hi, 8) == 0 and o.dequantize(0, lo, hi, 8) == lo
        if hi > lo:
            assert o.quantize(hi, lo, hi, 8) == 255
        xs = np.sort(rng.uniform(lo, hi, 64).astype(np.float32))
        codes = [o.quantize(float(x), lo, hi, 8) for x in xs]
        assert all(0 <= c <= 255 for c in codes)
        assert all(a <= b for a, b in zip(codes, codes[1:])), "codes not monotone"
        slack = 4 * float(_ulp(max(abs(lo), abs(hi))))
        for x, c in zip(xs, codes):
            assert abs(o.dequantize(c, lo, hi, 8) - float(x)) <= u / 2 + slack, (x, lo, hi)


# Published known-answer vectors of Philox4x32-10 (counter, key -> output),
# from the Random123 distribution that accompanies Salmon et al. (SC 2011).
PHILOX_KAT = [
    ((0, 0, 0, 0), (0, 0), (0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8)),
    ((0xFFFFFFFF,) * 4, (0xFFFFFFFF,) * 2, (0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD)),
    ((0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344), (0xA4093822, 0x299F31D0),
     (0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1)),
]


def check_philox_kat(o) -> None:
    for ctr, key, want in PHILOX_KAT:
        assert o.philox4x32_10(ctr, key) == want, (ctr, key)


def check_uniform_stream(o) -> None:
    seed = 0x0123456789ABCDEF
    # element i of tensor j at step t: top 24 bits of word i mod 4 of the
    # block at counter (i/4 low, i/4 high, j, t), key = the seed's two words
    for j, t, i in [(0, 1, 0), (3, 7, 5), (2, 2, 2 ** 33 + 6), (1, 1, 4095)]:
        out = o.philox4x32_10(((i >> 2) & 0xFFFFFFFF, i >> 34, j, t), (seed & 0xFFFFFFFF, seed >> 32))
        assert o.uniform_xi(seed, j, t, i) == (out[i & 3] >> 8) * 2.0 ** -24, (j, t, i)
    xs = np.array([o.uniform_xi(seed, 0, 1, i) for i in range(40000)])
    assert xs.min() >= 0.0 and xs.max() < 1.0
    assert np.array_equal(xs * 2 ** 24, np.floor(xs * 2 ** 24)), "not on the 2^-24 grid"
    assert abs(xs.mean() - 0.5) < 5 * math.sqrt(1 / 12 / xs.size)
    counts = np.bincount((xs * 16).astype(np.int64), minlength=16)
    chi2 = float(((counts - xs.size / 16) ** 2 / (xs.size / 16)).sum())
    assert chi2 < 44.3, chi2      # 15 degrees of freedom, upper 0.01% point
    base = [o.uniform_xi(seed, 0, 1, i) for i in range(64)]
    assert base != [o.uniform_xi(seed, 0, 2, i) for i in range(64)], "step not in the counter"
    assert base != [o.uniform_xi(seed, 1, 1, i) for i in range(64)], "tensor not in the counter"
    assert base != [o.uniform_xi(seed + 1, 0, 1, i) for i in range(64)]
    assert base != [o.uniform_xi(seed + (1 << 32), 0, 1, i) for i in range(64)]


def check_randomized_quantizer(o) -> None:
    rng = np.random.default_rng(21)
    K = 256
    xis = [(k + 0.5) / K for k in range(K)]
    for bits in (4, 8):
        L = 2 ** bits - 1
        for _ in range(30):
            lo, hi = np.sort(rng.standard_normal(2).astype(np.float32) * np.float32(10.0 ** rng.integers(-4, 2)))
            lo, hi = float(lo), float(hi)
            u = (hi - lo) / L
            slack = 8 * float(_ulp(max(abs(lo), abs(hi))))
            for x in rng.uniform(lo, hi, 6).astype(np.float32):
                codes = [o.quantize_randomized(float(x), lo, hi, xi, bits) for xi in xis]
                assert all(0 <= c <= L for c in codes)
                assert max(codes) - min(codes) <= 1, "a draw away from the two grid points around x"
                mean = float(np.mean([o.dequantize(c, lo, hi, bits) for c in codes]))
                assert abs(mean - float(x)) <= u / K + slack, ("biased", bits, float(x), lo, hi, mean)
            assert all(o.quantize_randomized(lo, lo, hi, xi, bits) == 0 for xi in (0.0, 0.5, 1 - 2 ** -24))
            if hi > lo:
                assert o.quantize_randomized(hi, lo, hi, 0.5, bits) == L
    # xi = 0 truncates; a grid point stays put for any xi below 1
    assert o.quantize_randomized(2.3, 0.0, 15.0, 0.0) == 2
    assert o.quantize_randomized(2.3, 0.0, 15.0, 0.75) == 3
    assert o.quantize_randomized(2.0, 0.0, 15.0, 1 - 2 ** -24) == 2
    assert o.quantize(3.0, 3.0, 3.0) == 0 and o.quantize_randomized(3.0, 3.0, 3.0, 0.9) == 0


def check_randomized_ef_unbiased(o) -> None:
    """Whole steps with randomized Q: averaged over seeds, the decoded error
    feedback after step 1 is the residual a - T_k(a) (Lemma 1), and each
    bucket meets the lemma's norm bound."""
    rng = np.random.default_rng(23)
    n, block, bucket, S = 512, 256, 64, 300
    g = rng.standard_normal(n).astype(np.float32)
    for bits in (4, 8):
        L = 2 ** bits - 1
        acc = np.zeros(n)
        codes0 = None
        for seed in range(S):
            st = o.tensor(n, block=block, bucket=bucket, density=0.05, window=2, rounding=1,
                          seed=seed, tensor=3, ef_bits=bits)
            st.step(np.zeros(n, np.float32), g, 1, 1e-3)
            dec = _decode(st.codes(), st.delta, st.Delta, bucket, L).astype(np.float64)
            acc += dec
            codes0 = st.codes() if codes0 is None else codes0
            r = g.astype(np.float64).copy()
            for q in range(st.nblocks):
                idx, _ = st.window_entries(0, q)
                r[q * block + idx.astype(np.int64)] = 0.0
            for b0 in range(0, n, bucket):
                x, xh = r[b0:b0 + bucket], dec[b0:b0 + bucket]
                lo, hi = x.min(), x.max()
                bound = math.sqrt(bucket - 2) / L * (hi - lo) / math.sqrt(hi * hi + lo * lo)
                assert np.linalg.norm(xh - x) <= bound * np.linalg.norm(x) * (1 + 1e-5), (bits, seed, b0)
        bidx = np.arange(n) // bucket
        u = (st.Delta[bidx].astype(np.float64) - st.delta[bidx]) / L
        assert np.all(np.abs(acc / S - r) <= 6 * u / (2 * math.sqrt(S)) + 1e-6), bits
        other = o.tensor(n, block=block, bucket=bucket, density=0.05, window=2, rounding=1,
                         seed=0, tensor=4, ef_bits=bits)
        other.step(np.zeros(n, np.float32), g, 1, 1e-3)
        assert not np.array_equal(other.codes(), codes0), "tensor number not in the stream"


def check_reconstruction_8bit(o) -> None:
    rng = np.random.default_rng(26)
    n, block, bucket = 2000, 256, 32
    st = o.tensor(n, block=block, bucket=bucket, density=0.02, window=3, ef_bits=8)
    theta = np.zeros(n, np.float32)
    for t in range(1, 5):
        g = rng.standard_normal(n).astype(np.float32)
        a = (g + _decode(st.codes(), st.delta, st.Delta, bucket, 255)).astype(np.float32)
        st.step(theta, g, t, 1e-3)
        rec = _decode(st.codes(), st.delta, st.Delta, bucket, 255).astype(np.float64)
        bidx = np.arange(n) // bucket
        bound = (st.Delta[bidx].astype(np.float64) - st.delta[bidx]) / 255 / 2
        bound += 4 * _ulp(np.maximum(np.abs(st.delta[bidx]), np.abs(st.Delta[bidx])))
        row = st.row_of_step(t)
        for q in range(st.nblocks):
            idx, val = st.window_entries(row, q)
            i = q * block + idx.astype(np.int64)
            rec[i] += val
            bound[i] += np.abs(val.astype(np.float64) - a[i]) + _ulp(a[i])
        assert np.all(np.abs(rec - a) <= bound), t


def check_topk_bruteforce(o) -> None:
    rng = np.random.default_rng(7)
    cases = [
        dict(n=1000, block=128, bucket=16, density=0.05),   # k 7, tail 104 -> 6
        dict(n=700, block=64, bucket=8, density=0.2),       # k 13, tail 60 -> 12
        dict(n=96, block=32, bucket=32, density=0.5),       # k 16
    ]
    for ci, case in enumerate(cases):
        for kind in ("normal", "ties", "zeros"):
            n = case["n"]
            if kind == "normal":
                g = rng.standard_normal(n).astype(np.float32)
            elif kind == "ties":
                g = (rng.integers(-3, 4, n) * rng.choice([1.0, 0.5], n)).astype(np.float32)
            else:
                g = np.zeros(n, np.float32)
                g[rng.integers(0, n, 5)] = -1.0
            for value_bf16 in (False, True):
                kw = {k: v for k, v in case.items() if k != "n"}
                st = o.tensor(n, window=3, value_bf16=value_bf16, **kw)
                theta = np.zeros(n, np.float32)
                st.step(theta, g, 1, 1e-3)
                for q in range(st.nblocks):
                    s0 = q * case["block"]
                    xb = g[s0:s0 + st.block_size(q)]
                    want = _brute_topk(xb, st.block_k(q))
                    idx, val = st.window_entries(0, q)
                    assert list(idx) == want, (ci, kind, q)
                    wv = xb[want]
                    if value_bf16:
                        wv = _bf16(wv)
                    assert np.array_equal(val.view(np.uint32), wv.view(np.uint32)), (ci, kind, q)


def check_k_per_block(o) -> None:
    """k = ceil(density * s) per block (the paper sizes k as ceil(d/100) for
    1% density), checked with exact rational arithmetic."""
    for s, dens in [(4096, "1/100"), (768, "1/100"), (3072, "1/100"), (3584, "1/100"),
                    (100, "1/100"), (1024, "1/100"), (65536, "1/20"), (12032, "1/20"),
                    (60, "1/20"), (4096, "1"), (7, "1/1000"), (200, "3/100")]:
        f = Fraction(dens)
        want = min(s, max(1, math.ceil(f * s)))
        assert o.block_k(s, float(f)) == want, (s, dens)
    # and the window holds exactly that many entries per block
    st = o.tensor(1000, block=128, bucket=16, density=0.05, window=2)
    st.step(np.zeros(1000, np.float32), np.ones(1000, np.float32), 1, 1e-3)
    assert st.K == 7 * 7 + math.ceil(Fraction(1, 20) * 104)


def check_contraction(o) -> None:
    rng = np.random.default_rng(8)
    n, block = 5000, 500
    g = (rng.standard_t(3, n) * 1e-2).astype(np.float32)
    st = o.tensor(n, block=block, bucket=50, density=0.03, window=2, value_bf16=False)
    st.step(np.zeros(n, np.float32), g, 1, 1e-3)
    for q in range(st.nblocks):
        a = g[q * block:(q + 1) * block].astype(np.float64)
        idx, _ = st.window_entries(0, q)
        r = a.copy()
        r[idx.astype(np.int64)] = 0.0
        k = st.block_k(q)
        assert (r ** 2).sum() <= (1 - k / a.size) * (a ** 2).sum() * (1 + 1e-12)


def check_ef_after_first_step(o) -> None:
    rng = np.random.default_rng(9)
    n, block, bucket = 1001, 128, 16          # odd n, 9-element tail bucket
    g = rng.standard_normal(n).astype(np.float32)
    st = o.tensor(n, block=block, bucket=bucket, density=0.05, window=4)
    st.step(np.zeros(n, np.float32), g, 1, 1e-3)
    r = g.copy()                               # residual a - T_k(a) at t = 1
    for q in range(st.nblocks):
        idx, _ = st.window_entries(0, q)
        r[q * block + idx.astype(np.int64)] = 0.0
    codes = st.codes()
    assert st.ef.size == (n + 1) // 2 and (st.ef[-1] >> 4) == 0
    for b in range(st.nbuckets):
        x = r[b * bucket:(b + 1) * bucket]
        lo, hi = np.float32(x.min()) + np.float32(0), np.float32(x.max()) + np.float32(0)
        assert st.delta[b].view(np.uint32) == lo.view(np.uint32), b
        assert st.Delta[b].view(np.uint32) == hi.view(np.uint32), b
        c = codes[b * bucket:(b + 1) * bucket]
        assert c[np.argmin(x)] == 0
        if hi > lo:
            assert c[np.argmax(x)] == 15


def check_reconstruction(o) -> None:
    rng = np.random.default_rng(10)
    n, block, bucket = 3000, 256, 32
    st = o.tensor(n, block=block, bucket=bucket, density=0.02, window=3)
    theta = np.zeros(n, np.float32)
    for t in range(1, 6):
        g = rng.standard_normal(n).astype(np.float32)
        a = (g + _decode(st.codes(), st.delta, st.Delta, bucket)).astype(np.float32)
        st.step(theta, g, t, 1e-3)
        rec = _decode(st.codes(), st.delta, st.Delta, bucket).astype(np.float64)
        bound = np.zeros(n)
        bidx = np.arange(n) // bucket
        bound += (st.Delta[bidx].astype(np.float64) - st.delta[bidx]) / 15 / 2
        bound += 4 * _ulp(np.maximum(np.abs(st.delta[bidx]), np.abs(st.Delta[bidx])))
        row = st.row_of_step(t)
        for q in range(st.nblocks):
            idx, val = st.window_entries(row, q)
            i = q * block + idx.astype(np.int64)
            rec[i] += val
            bound[i] += np.abs(val.astype(np.float64) - a[i]) + _ulp(a[i])
        assert np.all(np.abs(rec - a) <= bound), t


def _sliding(gs, beta, m, t):
    """Truncated bias-corrected EMA of g_1..g_t over the last m steps, built by
    a sliding recurrence S_t = beta*S_{t-1} + g_t - beta^m g_{t-m}."""
    S = np.zeros_like(gs[0])
    for s in range(1, t + 1):
        S = beta * S + gs[s - 1]
        if s - m >= 1:
            S = S - beta ** m * gs[s - m - 1]
    return (1 - beta) * S / (1 - beta ** t)


def check_density_one_is_adam(o) -> None:
    rng = np.random.default_rng(12)
    n, m = 300, 4
    st = o.tensor(n, block=64, bucket=16, density=1.0, window=m, value_bf16=False)
    theta = np.zeros(n, np.float32)
    gs = []
    m1 = np.zeros(n)
    v1 = np.zeros(n)
    for t in range(1, 10):
        g = rng.standard_normal(n).astype(np.float32)
        gs.append(g.astype(np.float64))
        st.step(theta, g, t, 1e-3)
        assert not st.ef.any() and not st.delta.any() and not st.Delta.any()
        mh, vh = st.moments(t)
        if t <= m:        # plain Adam: m_t = b1 m + (1-b1) g, bias-corrected
            m1 = BETA1 * m1 + (1 - BETA1) * gs[-1]
            v1 = BETA2 * v1 + (1 - BETA2) * gs[-1] ** 2
            want_m, want_v = m1 / (1 - BETA1 ** t), v1 / (1 - BETA2 ** t)
        else:
            want_m = _sliding(gs, BETA1, m, t)
            want_v = _sliding([x ** 2 for x in gs], BETA2, m, t)
        scale_m = sum(np.abs(x) for x in gs[-m:]) + 1e-30
        assert np.all(np.abs(mh - want_m) <= 1e-10 * scale_m), t
        assert np.allclose(vh, want_v, rtol=1e-10, atol=0), t


def check_first_step_closed_form(o) -> None:
    rng = np.random.default_rng(13)
    n, lr = 2000, 1e-3
    st = o.tensor(n, block=256, bucket=32, density=0.02, window=5)
    theta0 = (rng.standard_normal(n) * 0.02).astype(np.float32)
    g = (rng.standard_normal(n) * 1e-3).astype(np.float32)
    theta = theta0.copy()
    st.step(theta, g, 1, lr)
    want = theta0.copy()
    for q in range(st.nblocks):
        idx, val = st.window_entries(0, q)
        i = q * 256 + idx.astype(np.int64)
        V = val.astype(np.float64)
        want[i] = (theta0[i].astype(np.float64) - lr * V / (EPS + np.abs(V))).astype(np.float32)
        assert np.array_equal(val, _bf16(g[i]))
    assert np.array_equal(theta.view(np.uint32), want.view(np.uint32))


def check_window_one_closed_form(o) -> None:
    rng = np.random.default_rng(14)
    n = 1500
    st = o.tensor(n, block=500, bucket=50, density=0.05, window=1)
    theta = np.zeros(n, np.float32)
    for t in range(1, 6):
        st.step(theta, rng.standard_normal(n).astype(np.float32), t, 1e-3)
        mh, vh = st.moments(t)
        wm, wv = np.zeros(n), np.zeros(n)
        for q in range(st.nblocks):
            idx, val = st.window_entries(0, q)
            V = val.astype(np.float64)
            wm[q * 500 + idx.astype(np.int64)] = (1 - BETA1) / (1 - BETA1 ** t) * V
            wv[q * 500 + idx.astype(np.int64)] = (1 - BETA2) / (1 - BETA2 ** t) * V * V
        assert np.allclose(mh, wm, rtol=1e-12, atol=0), t
        assert np.allclose(vh, wv, rtol=1e-12, atol=0), t


def check_decay_exponents(o) -> None:
    """One spike per step at a fresh position; k = 1 per block keeps exactly
    that spike, so each live row contributes one known term beta^(t-s) V_s."""
    n, m = 64, 3
    pos = [5, 17, 29, 41, 53, 60, 2]
    st = o.tensor(n, block=64, bucket=16, density=1 / 64, window=m, value_bf16=False)
    theta = np.zeros(n, np.float32)
    rng = np.random.default_rng(15)
    spikes = {}
    for t in range(1, len(pos) + 1):
        g = (rng.standard_normal(n) * 1e-4).astype(np.float32)
        g[pos[t - 1]] = 10.0 + t
        st.step(theta, g, t, 1e-3)
        idx, val = st.window_entries(st.row_of_step(t), 0)
        assert list(idx) == [pos[t - 1]]
        spikes[t] = float(val[0])
        mh, vh = st.moments(t)
        want_m, want_v = np.zeros(n), np.zeros(n)
        for s in range(max(1, t - m + 1), t + 1):
            want_m[pos[s - 1]] = (1 - BETA1) / (1 - BETA1 ** t) * BETA1 ** (t - s) * spikes[s]
            want_v[pos[s - 1]] = (1 - BETA2) / (1 - BETA2 ** t) * BETA2 ** (t - s) * spikes[s] ** 2
        assert np.allclose(mh, want_m, rtol=1e-12, atol=0), t
        assert np.allclose(vh, want_v, rtol=1e-12, atol=0), t


def check_untouched_and_sparsity(o) -> None:
    rng = np.random.default_rng(16)
    n, block, m = 4096, 512, 3
    st = o.tensor(n, block=block, bucket=64, density=0.01, window=m)
    theta0 = (rng.standard_normal(n) * 0.02).astype(np.float32)
    theta = theta0.copy()
    for t in range(1, 7):
        before = theta.copy()
        st.step(theta, rng.standard_normal(n).astype(np.float32), t, 1e-3)
        live = np.zeros(n, bool)
        nlive = 0
        for s in range(max(1, t - m + 1), t + 1):
            for q in range(st.nblocks):
                idx, _ = st.window_entries(st.row_of_step(s), q)
                live[q * block + idx.astype(np.int64)] = True
                nlive += idx.size
        assert np.array_equal(theta[~live].view(np.uint32), before[~live].view(np.uint32))
        assert np.count_nonzero(theta != before) <= nlive


def check_weight_decay(o) -> None:
    rng = np.random.default_rng(17)
    n, lr, wd = 2048, 1e-2, 0.1
    st = o.tensor(n, block=1024, bucket=64, density=0.01, window=2, weight_decay=wd)
    theta0 = (rng.standard_normal(n) * 0.02).astype(np.float32)
    theta = theta0.copy()
    st.step(theta, rng.standard_normal(n).astype(np.float32), 1, lr)
    live = np.zeros(n, bool)
    for q in range(st.nblocks):
        idx, val = st.window_entries(0, q)
        live[q * 1024 + idx.astype(np.int64)] = True
    want = (theta0.astype(np.float64) * (1 - lr * wd)).astype(np.float32)
    assert np.array_equal(theta[~live], want[~live])
    assert not np.array_equal(theta[live], want[live])


def check_first_step_closed_form_bf16(o) -> None:
    """bf16 parameters: at t = 1, m-hat = V and v-hat = V^2, so every kept
    entry moves to theta_0 - eta*V/(eps + |V|), rounded once from the exact
    value to bf16; every other entry keeps its bits (lambda = 0)."""
    # the helper itself on two double-rounding traps
    assert _bf16_from_f64([1.0 + 2.0 ** -8 + 2.0 ** -40])[0] == 1.0 + 2.0 ** -7
    assert _bf16_from_f64([1.0 - 2.0 ** -9 - 2.0 ** -35])[0] == 1.0 - 2.0 ** -8
    rng = np.random.default_rng(27)
    n, block = 2000, 256
    cases = [
        # random bf16 parameters and gradients, the eps of Appendix B
        (_bf16(rng.standard_normal(n) * 0.02), (rng.standard_normal(n) * 1e-3).astype(np.float32),
         1e-3, EPS),
        # eps = 2^-100 (eps + |V| == |V| exactly for these V) and positive V:
        # a kept entry moves by exactly eta, and eta = 2^-9 + 2^-35 puts
        # 1 - eta just below the bf16 midpoint 1 - 2^-9, where one rounding
        # gives 1 - 2^-8 and a rounding through binary32 (onto the midpoint,
        # then to even) gives 1.0
        (np.ones(n, np.float32), (np.abs(rng.standard_normal(n)) + 0.1).astype(np.float32),
         2.0 ** -9 + 2.0 ** -35, 2.0 ** -100),
    ]
    for ci, (theta0, g, lr, eps) in enumerate(cases):
        st = o.tensor(n, block=block, bucket=32, density=0.02, window=5, param_bf16=True, eps=eps)
        theta = theta0.copy()
        st.step(theta, g, 1, lr)
        kept = np.zeros(n, bool)
        want = theta0.astype(np.float64)
        for q in range(st.nblocks):
            idx, val = st.window_entries(0, q)
            i = q * block + idx.astype(np.int64)
            kept[i] = True
            V = val.astype(np.float64)
            want[i] = theta0[i].astype(np.float64) - lr * (V / (eps + np.abs(V)))
        want = _bf16_from_f64(want)
        assert np.array_equal(theta.view(np.uint32), want.view(np.uint32)), ci
        assert np.array_equal(theta[~kept].view(np.uint32), theta0[~kept].view(np.uint32)), ci
        if ci == 1:
            assert np.all(theta[kept] == np.float32(1.0 - 2.0 ** -8))


# (n, B_d, B_q) with buckets that are not inside blocks: larger than the
# block and not a multiple of it, a multiple of it, and one bucket holding
# the whole tensor
SPANNING = [(1001, 64, 200), (640, 64, 192), (3000, 128, 1000), (300, 32, 100000)]


def _check_bucket_codes(st, r, bucket, levels=15):
    """delta/Delta of every bucket (tensor elements [c*B_q, (c+1)*B_q)) are
    the min/max of the residual r there; min -> code 0, max -> the top code,
    every element within half a step."""
    codes = st.codes()
    dec = _decode(codes, st.delta, st.Delta, bucket, levels).astype(np.float64)
    assert st.nbuckets == -(-r.size // bucket)
    for b in range(st.nbuckets):
        x = r[b * bucket:(b + 1) * bucket]
        lo, hi = np.float32(x.min()) + np.float32(0), np.float32(x.max()) + np.float32(0)
        assert st.delta[b].view(np.uint32) == lo.view(np.uint32), b
        assert st.Delta[b].view(np.uint32) == hi.view(np.uint32), b
        c = codes[b * bucket:(b + 1) * bucket]
        assert c[np.argmin(x)] == 0, b
        if hi > lo:
            assert c[np.argmax(x)] == levels, b
        u = (float(hi) - float(lo)) / levels
        slack = 4 * float(_ulp(max(abs(lo), abs(hi))))
        assert np.all(np.abs(dec[b * bucket:(b + 1) * bucket] - x) <= u / 2 + slack), b


def check_spanning_buckets_first_step(o) -> None:
    """Buckets spanning blocks, step 1: e = Q(g with g[I] = 0) with each
    tensor's buckets counted from its element 0."""
    rng = np.random.default_rng(28)
    for n, block, bucket in SPANNING:
        g = rng.standard_normal(n).astype(np.float32)
        st = o.tensor(n, block=block, bucket=bucket, density=0.05, window=3)
        st.step(np.zeros(n, np.float32), g, 1, 1e-3)
        r = g.copy()
        for q in range(st.nblocks):
            idx, _ = st.window_entries(0, q)
            assert list(idx) == _brute_topk(g[q * block:(q + 1) * block], st.block_k(q))
            r[q * block + idx.astype(np.int64)] = 0.0
        _check_bucket_codes(st, r, bucket)


def check_spanning_buckets_reconstruction(o) -> None:
    """Buckets spanning blocks over five steps: each step's accumulator a_t
    (decoded with the previous step's pairs) equals the next EF decoded with
    the new pairs plus the kept entries, within half a step (plus the bf16
    rounding of the kept values)."""
    rng = np.random.default_rng(29)
    for n, block, bucket in SPANNING:
        st = o.tensor(n, block=block, bucket=bucket, density=0.05, window=3)
        theta = np.zeros(n, np.float32)
        for t in range(1, 6):
            g = rng.standard_normal(n).astype(np.float32)
            a = (g + _decode(st.codes(), st.delta, st.Delta, bucket)).astype(np.float32)
            st.step(theta, g, t, 1e-3)
            r = a.copy()
            row = st.row_of_step(t)
            extra = np.zeros(n)
            for q in range(st.nblocks):
                idx, val = st.window_entries(row, q)
                i = q * block + idx.astype(np.int64)
                assert list(idx) == _brute_topk(a[q * block:(q + 1) * block], st.block_k(q)), (n, t, q)
                r[i] = 0.0
                extra[i] = np.abs(val.astype(np.float64) - a[i]) + _ulp(a[i])
            _check_bucket_codes(st, r, bucket)
            rec = _decode(st.codes(), st.delta, st.Delta, bucket).astype(np.float64)
            for q in range(st.nblocks):
                idx, val = st.window_entries(row, q)
                rec[q * block + idx.astype(np.int64)] += val
            bidx = np.arange(n) // bucket
            bound = (st.Delta[bidx].astype(np.float64) - st.delta[bidx]) / 15 / 2
            bound += 4 * _ulp(np.maximum(np.abs(st.delta[bidx]), np.abs(st.Delta[bidx]))) + extra
            assert np.all(np.abs(rec - a) <= bound), (n, t)


def check_spanning_buckets_lemma1(o) -> None:
    """Randomized rounding with buckets spanning blocks: every bucket of the
    first step's error feedback meets Lemma 1's norm bound, and the decoded
    EF averaged over seeds is the residual."""
    rng = np.random.default_rng(30)
    n, block, bucket, S = 700, 64, 200, 120
    g = rng.standard_normal(n).astype(np.float32)
    acc = np.zeros(n)
    for seed in range(S):
        st = o.tensor(n, block=block, bucket=bucket, density=0.05, window=2, rounding=1, seed=seed, tensor=1)
        st.step(np.zeros(n, np.float32), g, 1, 1e-3)
        dec = _decode(st.codes(), st.delta, st.Delta, bucket).astype(np.float64)
        acc += dec
        r = g.astype(np.float64).copy()
        for q in range(st.nblocks):
            idx, _ = st.window_entries(0, q)
            r[q * block + idx.astype(np.int64)] = 0.0
        for b0 in range(0, n, bucket):
            x, xh = r[b0:b0 + bucket], dec[b0:b0 + bucket]
            lo, hi = x.min(), x.max()
            assert st.delta[b0 // bucket] == np.float32(lo) and st.Delta[b0 // bucket] == np.float32(hi)
            bound = math.sqrt(x.size - 2) / 15 * (hi - lo) / math.sqrt(hi * hi + lo * lo)
            assert np.linalg.norm(xh - x) <= bound * np.linalg.norm(x) * (1 + 1e-5), (seed, b0)
    bidx = np.arange(n) // bucket
    u = (st.Delta[bidx].astype(np.float64) - st.delta[bidx]) / 15
    assert np.all(np.abs(acc / S - r) <= 6 * u / (2 * math.sqrt(S)) + 1e-6)


ALL_CHECKS = [
    check_round_bf16,
    check_quantizer,
    check_topk_bruteforce,
    check_k_per_block,
    check_contraction,
    check_ef_after_first_step,
    check_reconstruction,
    check_density_one_is_adam,
    check_first_step_closed_form,
    check_window_one_closed_form,
    check_decay_exponents,
    check_untouched_and_sparsity,
    check_weight_decay,
    check_quantizer_8bit,
    check_philox_kat,
    check_uniform_stream,
    check_randomized_quantizer,
    check_randomized_ef_unbiased,
    check_reconstruction_8bit,
    check_first_step_closed_form_bf16,
    check_spanning_buckets_first_step,
    check_spanning_buckets_reconstruction,
    check_spanning_buckets_lemma1,
]
