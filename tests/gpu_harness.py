"""Drives libmicroadam (through its C ABI binding) and the CPU oracle on the
same seeded inputs and compares them after every step.

Bit-exact: the EF codes (4- or 8-bit, nearest or randomized rounding), the
bucket (delta, Delta) pairs and every live window row (indices and bf16 /
float32 values).  Within tolerance: the
parameters and the window moments, which the kernel computes in binary32 and
the oracle in binary64.  Tolerances (relative, per element):
  parameters  |x - y| <= tol * max(|y|, lr)   tol 1e-5 for float32 storage,
                                              2e-2 for bf16 storage, and for
              bf16 also |x - y| <= one bf16 ulp of y (exact_fraction records
              the share of bit-identical elements)
  m-hat       |x - y| <= 1e-5 * c1 * sum_r beta1^r |V_r|   (summation bound)
  v-hat       |x - y| <= 1e-5 * |y|
The oracle's parameters are reset to the GPU's before each step, so each
comparison covers exactly one step.

Large workloads are checked on sampled Top-K blocks: blocks share nothing, so
the oracle runs each sampled block as a tensor of its own over all steps.
"""
from __future__ import annotations

import math

import numpy as np
import torch

import oracle
import paper_2405_15593_amd as ma
from paper_2405_15593_amd import workloads as wl


def _f32(t: torch.Tensor) -> np.ndarray:
    return t.detach().float().cpu().numpy().astype(np.float32)


def bf16_ulp(y: np.ndarray) -> np.ndarray:
    """Spacing of the bf16 values in the binade of each y (8 significant
    bits; subnormal spacing 2^-133 at the bottom)."""
    _, e = np.frexp(np.abs(y))            # |y| in [2^(e-1), 2^e)
    e = np.where(y == 0, -200, e)
    return np.ldexp(1.0, np.maximum(e - 8, -133)).astype(np.float64)


class Unit:
    """Blocks [q0, q1) of tensor j, run by the oracle as a tensor of its own."""

    def __init__(self, o, j, q0, q1, numel, block, okw):
        self.j, self.q0, self.q1 = j, q0, q1
        self.e0 = q0 * block
        self.e1 = min(numel, q1 * block)
        # the randomized rounding's stream is keyed by the tensor number and
        # the element's place in the whole tensor
        self.state = o.tensor(self.e1 - self.e0, block=block, tensor=j, offset=self.e0, **okw)


class GpuOracleRun:
    def __init__(self, numels, *, param_dtype=torch.float32, grad_dtype=torch.float32,
                 grad_dist="normal", grad_scale=1.0, lr=1e-3, seed=0, sample=None,
                 density=0.01, window=10, bucket=64, block=4096, value_f32=False,
                 beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.0, ef_bits=4,
                 ef_rounding=0, ef_seed=0, degenerate=False, fused=0, device="cuda"):
        self.numels = list(numels)
        self.lr = lr
        self.device = torch.device(device)
        self.grad_dist, self.grad_scale, self.grad_dtype = grad_dist, grad_scale, grad_dtype
        self.seed = seed
        self.block, self.bucket, self.window = block, bucket, window
        self.cfg = ma.make_config(density=density, beta1=beta1, beta2=beta2, eps=eps, lr=lr,
                                  weight_decay=weight_decay, window=window, ef_bucket=bucket,
                                  topk_block=block, ef_bits=ef_bits, ef_rounding=ef_rounding, seed=ef_seed,
                                  fused=fused,
                                  window_value_dtype=ma.MICROADAM_F32 if value_f32 else ma.MICROADAM_BF16)
        self.ef_bits = ef_bits
        self.degenerate = degenerate  # inputs whose codes, rows or updates may all be zero
        self.params = [wl.draw(n, "normal", 0.02, seed + 7919 * (j + 1), self.device, param_dtype)
                       for j, n in enumerate(self.numels)]
        self.opt = ma.MicroAdam(self.params, self.cfg)
        self.o = oracle.default()
        okw = dict(bucket=bucket, window=window, density=density, value_bf16=not value_f32,
                   param_bf16=param_dtype == torch.bfloat16, beta1=beta1, beta2=beta2, eps=eps,
                   weight_decay=weight_decay, ef_bits=ef_bits, rounding=ef_rounding, seed=ef_seed)
        self.value_f32 = value_f32
        self.units: list[Unit] = []
        for j, n in enumerate(self.numels):
            nb = -(-n // block)
            if sample is None:
                self.units.append(Unit(self.o, j, 0, nb, n, block, okw))
            else:
                for q in sample(j, nb):
                    self.units.append(Unit(self.o, j, q, q + 1, n, block, okw))
        self.t = 0
        self.betas = (beta1, beta2)
        self.exact_fraction = 1.0
        self.exact_history: list[float] = []

    # ---------------------------------------------------------------- steps
    def grads(self, t):
        return [wl.draw(n, self.grad_dist, self.grad_scale, wl.grad_seed(t, j, self.seed),
                        self.device, self.grad_dtype) for j, n in enumerate(self.numels)]

    def step(self, check_moments=True):
        t = self.t + 1
        g = self.grads(t)
        theta_before = {}
        for u in self.units:
            theta_before[id(u)] = _f32(self.params[u.j][u.e0:u.e1])
        self.opt.step(g)
        torch.cuda.synchronize()
        for u in self.units:
            th = theta_before[id(u)].copy()
            u.state.step(th, _f32(g[u.j][u.e0:u.e1]), t, self.lr)
            u.theta_ref = th
            u.theta_before = theta_before[id(u)]
        self.t = t
        self.check_state(t)
        self.check_params()
        if check_moments:
            self.check_moments(t)

    # ------------------------------------------------------ GPU state reads
    def _read(self, off, nbytes) -> np.ndarray:
        return self.opt.state_view[off:off + nbytes].cpu().numpy()

    def _block_elems(self, lay, q: int) -> int:
        return min(self.block, lay.numel - q * self.block)

    def gpu_codes(self, u: Unit):
        """Codes of the unit's elements and the raw bytes of its last block."""
        lay = self.opt.layout(u.j)
        parts, raw = [], None
        for q in range(u.q0, u.q1):
            n = self._block_elems(lay, q)
            if self.ef_bits == 8:
                raw = self._read(lay.ef_plane + lay.block_number(q) * lay.ef_stride, n)
                parts.append(raw.copy())
                continue
            raw = self._read(lay.ef_plane + lay.block_number(q) * lay.ef_stride, (n + 1) // 2)
            c = np.empty(2 * raw.size, np.uint8)
            c[0::2] = raw & 0x0F
            c[1::2] = raw >> 4
            parts.append(c[:n])
        return np.concatenate(parts), raw

    def gpu_stats(self, u: Unit):
        lay = self.opt.layout(u.j)
        if lay.bucket_table_bytes:
            # buckets spanning blocks: the tensor's pairs in the table of step t
            assert u.q0 == 0 and u.q1 == lay.num_blocks, "buckets spanning blocks need whole tensors"
            off = lay.stats_plane + (self.t % 2) * lay.bucket_table_bytes
            raw = self._read(off, 8 * lay.num_buckets).view(np.float32).reshape(-1, 2)
            return raw[:, 0].copy(), raw[:, 1].copy()
        lo, hi = [], []
        for q in range(u.q0, u.q1):
            nb = -(-self._block_elems(lay, q) // self.bucket)
            off = lay.stats_plane + lay.block_number(q) * lay.stats_stride
            raw = self._read(off, 8 * nb).view(np.float32).reshape(nb, 2)
            lo.append(raw[:, 0])
            hi.append(raw[:, 1])
        return np.concatenate(lo), np.concatenate(hi)

    def gpu_row(self, u: Unit, q: int, slot: int):
        """(indices, values) of block q (tensor-relative) in row slot `slot`."""
        lay = self.opt.layout(u.j)
        kq = lay.k_last if q == lay.num_blocks - 1 else lay.k_full
        eb = lay.entry_bytes
        off = lay.window_plane + lay.block_number(q) * lay.window_stride + slot * kq * eb
        raw = self._read(off, kq * eb)
        if eb == 4:
            w = raw.view(np.uint32)
            return (w & 0xFFFF).astype(np.uint16), (w & 0xFFFF0000).view(np.float32)
        w = raw.view(np.uint32).reshape(kq, 2)
        return w[:, 0].astype(np.uint16), w[:, 1].copy().view(np.float32)

    # ------------------------------------------------------------ checks
    def check_state(self, t):
        nonzero_codes = nonzero_vals = 0
        for u in self.units:
            st = u.state
            codes, raw = self.gpu_codes(u)
            nonzero_codes += int(np.count_nonzero(codes))
            nonzero_vals += int(np.count_nonzero(st.win_val))
            bad = np.nonzero(codes != st.codes())[0]
            assert bad.size == 0, (f"EF codes differ: tensor {u.j} block {u.q0} t={t}: "
                                   f"first at element {bad[0]}: gpu {codes[bad[0]]} oracle {st.codes()[bad[0]]}")
            if self.ef_bits == 4 and (u.e1 - u.e0) % 2 == 1:
                assert (raw[-1] >> 4) == 0, "odd tail nibble not zero"
            lo, hi = self.gpu_stats(u)
            assert np.array_equal(lo.view(np.uint32), st.delta.view(np.uint32)), f"delta differs t={t} tensor {u.j}"
            assert np.array_equal(hi.view(np.uint32), st.Delta.view(np.uint32)), f"Delta differs t={t} tensor {u.j}"
            for s in range(max(1, t - self.window + 1), t + 1):
                slot = (s - 1) % self.window
                for qq in range(u.q1 - u.q0):
                    gi, gv = self.gpu_row(u, u.q0 + qq, slot)
                    oi, ov = st.window_entries(slot, qq)
                    assert np.array_equal(gi, oi), (f"window indices differ: tensor {u.j} block "
                                                    f"{u.q0 + qq} row of step {s} at t={t}")
                    assert np.array_equal(gv.view(np.uint32), ov.view(np.uint32)), (
                        f"window values differ: tensor {u.j} block {u.q0 + qq} row of step {s} at t={t}")
        # the comparison must have looked at real data
        if not self.degenerate:
            assert nonzero_vals > 0, "no window value compared"
            if self.cfg.density < 1.0:
                assert nonzero_codes > 0, "no EF code compared"

    def check_params(self):
        """Parameters within tol * max(|y|, lr); bf16 parameters also within one
        bf16 ulp of the oracle's: both round the same update to bf16, the kernel
        from binary32 and the oracle from binary64, so they can differ only
        where the exact value lies within a few binary32 ulps of a bf16
        midpoint.  The fraction of bit-identical elements is recorded."""
        bf16_params = self.params[0].dtype == torch.bfloat16
        tol = 2e-2 if bf16_params else 1e-5
        changed = same = total = 0
        for u in self.units:
            got = _f32(self.params[u.j][u.e0:u.e1]).astype(np.float64)
            ref = u.theta_ref.astype(np.float64)
            changed += int(np.count_nonzero(got != u.theta_before))
            same += int(np.count_nonzero(got == ref))
            total += got.size
            lim = tol * np.maximum(np.abs(ref), self.lr)
            bad = np.nonzero(np.abs(got - ref) > lim)[0]
            assert bad.size == 0, (f"params differ: tensor {u.j} block {u.q0} element {bad[0]}: "
                                   f"gpu {got[bad[0]]!r} oracle {ref[bad[0]]!r}")
            if bf16_params:
                ulp = bf16_ulp(ref)
                bad = np.nonzero(np.abs(got - ref) > ulp)[0]
                assert bad.size == 0, (f"bf16 params more than one bf16 ulp apart: tensor {u.j} block {u.q0} "
                                       f"element {bad[0]}: gpu {got[bad[0]]!r} oracle {ref[bad[0]]!r}")
        assert changed > 0 or self.degenerate, "the step changed no parameter"
        self.exact_fraction = same / max(total, 1)
        self.exact_history.append(self.exact_fraction)

    def check_moments(self, t):
        b1, b2 = self.betas
        c1 = (1 - b1) / (1 - b1 ** t)
        # dense moments of one tensor at a time, on the device; only the
        # units' slices come to the host
        by_tensor = {}
        for u in self.units:
            by_tensor.setdefault(u.j, []).append(u)
        slices = {}
        for j, units in by_tensor.items():
            dm, dv = self.opt.debug_moments(j)
            for u in units:
                slices[id(u)] = (_f32(dm[u.e0:u.e1]), _f32(dv[u.e0:u.e1]))
            del dm, dv
        for u in self.units:
            gm, gv = slices[id(u)]
            gm, gv = gm.astype(np.float64), gv.astype(np.float64)
            rm, rv = u.state.moments(t)
            scale = np.zeros_like(rm)
            for s in range(max(1, t - self.window + 1), t + 1):
                slot = (s - 1) % self.window
                for qq in range(u.q1 - u.q0):
                    idx, val = u.state.window_entries(slot, qq)
                    np.add.at(scale, qq * self.block + idx.astype(np.int64),
                              c1 * b1 ** (t - s) * np.abs(val.astype(np.float64)))
            assert np.all(np.abs(gm - rm) <= 1e-5 * scale + 1e-30), f"m-hat differs at t={t} tensor {u.j}"
            assert np.all(np.abs(gv - rv) <= 1e-5 * np.abs(rv) + 1e-30), f"v-hat differs at t={t} tensor {u.j}"
