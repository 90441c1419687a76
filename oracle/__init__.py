"""MicroAdam CPU oracle -- TEST INFRASTRUCTURE ONLY.

A ctypes front end over ``microadam_oracle.c``: a plain, slow, single-threaded
CPU statement of one MicroAdam step (Algorithms 1, 2 and 4, Section 3.1 and,
as an option, the randomized quantizer of Lemma 1, of the MicroAdam paper).
Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  It shares no code
with the HIP path and must never be used to produce a product result.

State is held in the oracle's own layout (see the C file's header):
    ef       uint8[(n+1)//2]  4-bit codes, element 2j in the low nibble
             uint8[n]         (ef_bits = 8) one code per byte
    delta    float32[nb]      bucket minimum   (nb = ceil(n / bucket))
    Delta    float32[nb]      bucket maximum
    win_idx  uint16[m, K]     window rows of block-relative indices
    win_val  float32[m, K]    window rows of values (bf16-exact if value_bf16)
Block q's entries occupy columns [q*k_full, q*k_full + k_q) of every row.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(_HERE, "microadam_oracle.c")
LIBRARY = os.path.join(_HERE, "libmicroadam_oracle.so")
CFLAGS = ["-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
          "-fno-fast-math", "-frounding-math", "-Wall", "-Wextra"]


def build(source: str = SOURCE, out: str = LIBRARY) -> str:
    """Compile the oracle with gcc (no FMA contraction, no fast-math)."""
    tmp = f"{out}.{os.getpid()}.tmp"  # concurrent builds (test workers) do not share a temporary
    cmd = ["gcc", *CFLAGS, "-o", tmp, source, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


class _Cfg(ctypes.Structure):
    _fields_ = [
        ("n", ctypes.c_int64),
        ("block", ctypes.c_int32),
        ("bucket", ctypes.c_int32),
        ("window", ctypes.c_int32),
        ("value_bf16", ctypes.c_int32),
        ("param_bf16", ctypes.c_int32),
        ("ef_bits", ctypes.c_int32),
        ("density", ctypes.c_double),
        ("beta1", ctypes.c_double),
        ("beta2", ctypes.c_double),
        ("eps", ctypes.c_double),
        ("weight_decay", ctypes.c_double),
        ("rounding", ctypes.c_int32),
        ("tensor", ctypes.c_int32),
        ("seed", ctypes.c_uint64),
        ("offset", ctypes.c_int64),
    ]


def _ptr(a: np.ndarray, ctype):
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(ctypes.POINTER(ctype))


class Oracle:
    """Handle on one compiled oracle library (the default one, or a variant
    built from another source file by a test)."""

    def __init__(self, path: str = LIBRARY):
        if not os.path.exists(path):
            if path != LIBRARY:
                raise FileNotFoundError(path)
            build()
        lib = ctypes.CDLL(path)
        P = ctypes.POINTER
        lib.oracle_block_k.argtypes = [ctypes.c_int64, ctypes.c_double]
        lib.oracle_block_k.restype = ctypes.c_int64
        for f in ("oracle_num_blocks", "oracle_num_buckets", "oracle_row_width"):
            getattr(lib, f).argtypes = [P(_Cfg)]
            getattr(lib, f).restype = ctypes.c_int64
        lib.oracle_step.argtypes = [
            P(_Cfg), ctypes.c_int64, ctypes.c_double, P(ctypes.c_float),
            P(ctypes.c_float), P(ctypes.c_uint8), P(ctypes.c_float),
            P(ctypes.c_float), P(ctypes.c_uint16), P(ctypes.c_float),
            ctypes.c_int64, ctypes.c_int64]
        lib.oracle_step.restype = ctypes.c_int
        lib.oracle_moments.argtypes = [
            P(_Cfg), ctypes.c_int64, P(ctypes.c_uint16), P(ctypes.c_float),
            ctypes.c_int64, ctypes.c_int64, P(ctypes.c_double), P(ctypes.c_double)]
        lib.oracle_moments.restype = None
        lib.oracle_round_bf16.argtypes = [ctypes.c_double]
        lib.oracle_round_bf16.restype = ctypes.c_float
        lib.oracle_dequantize.argtypes = [ctypes.c_uint, ctypes.c_float, ctypes.c_float, ctypes.c_int]
        lib.oracle_dequantize.restype = ctypes.c_float
        lib.oracle_quantize.argtypes = [ctypes.c_float, ctypes.c_float, ctypes.c_float, ctypes.c_int]
        lib.oracle_quantize.restype = ctypes.c_uint
        lib.oracle_quantize_randomized.argtypes = [ctypes.c_float, ctypes.c_float, ctypes.c_float,
                                                   ctypes.c_int, ctypes.c_float]
        lib.oracle_quantize_randomized.restype = ctypes.c_uint
        lib.oracle_philox4x32_10.argtypes = [P(ctypes.c_uint32), ctypes.c_uint32, ctypes.c_uint32,
                                             P(ctypes.c_uint32)]
        lib.oracle_philox4x32_10.restype = None
        lib.oracle_uniform_xi.argtypes = [ctypes.c_uint64, ctypes.c_int32, ctypes.c_int64, ctypes.c_int64]
        lib.oracle_uniform_xi.restype = ctypes.c_float
        self.lib = lib

    def block_k(self, s: int, density: float) -> int:
        return int(self.lib.oracle_block_k(int(s), float(density)))

    def round_bf16(self, x: float) -> float:
        return float(self.lib.oracle_round_bf16(float(x)))

    def quantize(self, x: float, lo: float, hi: float, bits: int = 4) -> int:
        return int(self.lib.oracle_quantize(x, lo, hi, bits))

    def quantize_randomized(self, x: float, lo: float, hi: float, xi: float, bits: int = 4) -> int:
        return int(self.lib.oracle_quantize_randomized(x, lo, hi, bits, xi))

    def dequantize(self, code: int, lo: float, hi: float, bits: int = 4) -> float:
        return float(self.lib.oracle_dequantize(code, lo, hi, bits))

    def philox4x32_10(self, ctr, key) -> tuple:
        c = (ctypes.c_uint32 * 4)(*[int(x) & 0xFFFFFFFF for x in ctr])
        out = (ctypes.c_uint32 * 4)()
        self.lib.oracle_philox4x32_10(c, int(key[0]) & 0xFFFFFFFF, int(key[1]) & 0xFFFFFFFF, out)
        return tuple(int(x) for x in out)

    def uniform_xi(self, seed: int, tensor: int, t: int, i: int) -> float:
        return float(self.lib.oracle_uniform_xi(int(seed), int(tensor), int(t), int(i)))

    def tensor(self, n: int, **kw) -> "TensorState":
        return TensorState(self, n, **kw)


class TensorState:
    """The MicroAdam optimizer state of one parameter tensor, on the host."""

    def __init__(self, oracle: Oracle, n: int, *, block: int = 4096,
                 bucket: int = 64, window: int = 10, density: float = 0.01,
                 value_bf16: bool = True, param_bf16: bool = False,
                 beta1: float = 0.9, beta2: float = 0.999, eps: float = 1e-8,
                 weight_decay: float = 0.0, ef_bits: int = 4, rounding: int = 0,
                 seed: int = 0, tensor: int = 0, offset: int = 0):
        self.o = oracle
        self.cfg = _Cfg(n=n, block=block, bucket=bucket, window=window,
                        value_bf16=int(value_bf16), param_bf16=int(param_bf16),
                        ef_bits=int(ef_bits), density=density, beta1=beta1, beta2=beta2,
                        eps=eps, weight_decay=weight_decay, rounding=int(rounding),
                        tensor=int(tensor), seed=int(seed), offset=int(offset))
        self.ef_bits = int(ef_bits)
        lib = oracle.lib
        c = ctypes.byref(self.cfg)
        self.n = n
        self.nblocks = int(lib.oracle_num_blocks(c))
        self.nbuckets = int(lib.oracle_num_buckets(c))
        self.K = int(lib.oracle_row_width(c))
        self.k_full = oracle.block_k(block, density)
        self.ef = np.zeros(n if ef_bits == 8 else (n + 1) // 2, np.uint8)
        self.delta = np.zeros(self.nbuckets, np.float32)
        self.Delta = np.zeros(self.nbuckets, np.float32)
        self.win_idx = np.zeros((window, self.K), np.uint16)
        self.win_val = np.zeros((window, self.K), np.float32)

    # -- geometry ---------------------------------------------------------
    def block_size(self, q: int) -> int:
        return min(self.cfg.block, self.n - q * self.cfg.block)

    def block_k(self, q: int) -> int:
        return self.o.block_k(self.block_size(q), self.cfg.density)

    def block_slot(self, q: int) -> int:
        return q * self.k_full

    def row_of_step(self, s: int) -> int:
        return (s - 1) % self.cfg.window

    def window_entries(self, row: int, q: int):
        """(block-relative indices, values) of block q in window row `row`."""
        lo, k = self.block_slot(q), self.block_k(q)
        return self.win_idx[row, lo:lo + k].copy(), self.win_val[row, lo:lo + k].copy()

    def codes(self) -> np.ndarray:
        """The codes, one per element."""
        if self.ef_bits == 8:
            return self.ef.copy()
        c = np.empty(2 * self.ef.size, np.uint8)
        c[0::2] = self.ef & 0x0F
        c[1::2] = self.ef >> 4
        return c[: self.n]

    # -- the method -------------------------------------------------------
    def step(self, theta: np.ndarray, grad: np.ndarray, t: int, lr: float,
             q0: int = 0, q1: int | None = None) -> None:
        """One MicroAdam step at step t over blocks [q0, q1); `theta` is
        float32 and updated in place, `grad` is float32."""
        assert theta.dtype == np.float32 and grad.dtype == np.float32
        assert theta.size == self.n and grad.size == self.n
        q1 = self.nblocks if q1 is None else q1
        rc = self.o.lib.oracle_step(
            ctypes.byref(self.cfg), int(t), float(lr),
            _ptr(theta, ctypes.c_float), _ptr(grad, ctypes.c_float),
            _ptr(self.ef, ctypes.c_uint8), _ptr(self.delta, ctypes.c_float),
            _ptr(self.Delta, ctypes.c_float), _ptr(self.win_idx, ctypes.c_uint16),
            _ptr(self.win_val, ctypes.c_float), int(q0), int(q1))
        if rc != 0:
            raise ValueError(f"oracle_step rejected the configuration (rc={rc})")

    def moments(self, t: int, q0: int = 0, q1: int | None = None):
        """Dense binary64 (m_hat, v_hat) of the current window, blocks [q0, q1)."""
        q1 = self.nblocks if q1 is None else q1
        lo = q0 * self.cfg.block
        hi = min(self.n, q1 * self.cfg.block)
        mh = np.zeros(hi - lo, np.float64)
        vh = np.zeros(hi - lo, np.float64)
        self.o.lib.oracle_moments(
            ctypes.byref(self.cfg), int(t), _ptr(self.win_idx, ctypes.c_uint16),
            _ptr(self.win_val, ctypes.c_float), int(q0), int(q1),
            _ptr(mh, ctypes.c_double), _ptr(vh, ctypes.c_double))
        return mh, vh


_DEFAULT: Oracle | None = None


def default() -> Oracle:
    global _DEFAULT
    if _DEFAULT is None:
        _DEFAULT = Oracle()
    return _DEFAULT
