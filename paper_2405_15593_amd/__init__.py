"""MicroAdam optimizer step for AMD Instinct MI355X (gfx950).

A thin ctypes binding over ``libmicroadam.so`` (C ABI in ``include/microadam.h``).
Functions keep the C names and only marshal arguments; every step of the
method runs in the library's HIP kernels.  PyTorch supplies device memory and
streams (``MicroAdam`` below allocates the state buffer as a uint8 tensor).

Loading fails loudly when the library has not been built: there is no CPU
fallback.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Sequence

_PKG = os.path.dirname(os.path.abspath(__file__))
LIBRARY = os.path.join(_PKG, "libmicroadam.so")

MICROADAM_OK = 0
MICROADAM_ERR_INVALID_ARG = -1
MICROADAM_ERR_UNSUPPORTED = -2
MICROADAM_ERR_SHAPE = -3
MICROADAM_ERR_STATE_SIZE = -4
MICROADAM_ERR_HIP = -5
MICROADAM_ERR_NO_MEMORY = -6

MICROADAM_F32 = 0
MICROADAM_BF16 = 1
MICROADAM_ROUND_NEAREST = 0
MICROADAM_ROUND_RANDOMIZED = 1


class microadam_config(ctypes.Structure):
    _fields_ = [
        ("density", ctypes.c_double),
        ("beta1", ctypes.c_double),
        ("beta2", ctypes.c_double),
        ("eps", ctypes.c_double),
        ("lr", ctypes.c_double),
        ("weight_decay", ctypes.c_double),
        ("window", ctypes.c_int32),
        ("ef_bits", ctypes.c_int32),
        ("ef_bucket", ctypes.c_int32),
        ("topk_block", ctypes.c_int32),
        ("window_value_dtype", ctypes.c_int32),
        ("ef_rounding", ctypes.c_int32),
        ("seed", ctypes.c_uint64),
        ("fused", ctypes.c_int32),
        ("reserved", ctypes.c_int32),
    ]


class microadam_layout(ctypes.Structure):
    _fields_ = [
        ("numel", ctypes.c_int64),
        ("num_blocks", ctypes.c_int64),
        ("num_buckets", ctypes.c_int64),
        ("k_full", ctypes.c_int32),
        ("k_last", ctypes.c_int32),
        ("entry_bytes", ctypes.c_int32),
        ("reserved", ctypes.c_int32),
        ("first_block", ctypes.c_int64),
        ("last_block", ctypes.c_int64),
        ("ef_plane", ctypes.c_uint64),
        ("ef_stride", ctypes.c_uint64),
        ("stats_plane", ctypes.c_uint64),
        ("stats_stride", ctypes.c_uint64),
        ("window_plane", ctypes.c_uint64),
        ("window_stride", ctypes.c_uint64),
        ("bucket_table_bytes", ctypes.c_uint64),
    ]

    def block_number(self, q: int) -> int:
        """Global number of the tensor's block q."""
        return self.last_block if q == self.num_blocks - 1 else self.first_block + q


# every symbol include/microadam.h declares
EXPORTS = (
    "microadam_state_bytes", "microadam_init", "microadam_step", "microadam_destroy",
    "microadam_get_step", "microadam_set_step", "microadam_tensor_layout",
    "microadam_debug_moments", "microadam_step_kernels", "microadam_set_profiling", "microadam_kernel_times",
    "microadam_kernel_times_total", "microadam_step_noalloc", "microadam_error_string",
    "microadam_last_error",
)


class MicroAdamError(RuntimeError):
    def __init__(self, code: int, where: str, detail: str):
        super().__init__(f"{where}: {detail} (code {code})")
        self.code = code


_lib = None


def load(path: str = LIBRARY):
    """Loads libmicroadam.so; raises if it is not built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built: run `python -c 'import __graft_entry__ as g; g.build()'`")
    lib = ctypes.CDLL(path)
    P = ctypes.POINTER
    vp, i32, i64, u64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64
    lib.microadam_state_bytes.argtypes = [P(microadam_config), P(i64), i32, P(u64)]
    lib.microadam_init.argtypes = [P(microadam_config), P(i64), i32, i32, i32, vp, u64, vp, P(vp)]
    lib.microadam_step.argtypes = [vp, P(vp), P(vp), i32, ctypes.c_double, vp]
    lib.microadam_destroy.argtypes = [vp]
    lib.microadam_get_step.argtypes = [vp]
    lib.microadam_get_step.restype = i64
    lib.microadam_set_step.argtypes = [vp, i64]
    lib.microadam_tensor_layout.argtypes = [vp, i32, P(microadam_layout)]
    lib.microadam_debug_moments.argtypes = [vp, i32, vp, vp, vp]
    lib.microadam_step_kernels.argtypes = [vp]
    lib.microadam_step_noalloc.argtypes = [P(microadam_config), P(i64), i32, i32, i32, vp, u64, i64, P(vp), P(vp),
                                           ctypes.c_double, vp]
    lib.microadam_set_profiling.argtypes = [vp, i32]
    lib.microadam_kernel_times.argtypes = [vp, P(ctypes.c_float)]
    lib.microadam_kernel_times_total.argtypes = [vp, P(ctypes.c_float), P(i64)]
    lib.microadam_error_string.argtypes = [ctypes.c_int]
    lib.microadam_error_string.restype = ctypes.c_char_p
    lib.microadam_last_error.argtypes = []
    lib.microadam_last_error.restype = ctypes.c_char_p
    for f in ("microadam_state_bytes", "microadam_init", "microadam_step", "microadam_destroy",
              "microadam_set_step", "microadam_tensor_layout", "microadam_debug_moments",
              "microadam_step_kernels", "microadam_set_profiling", "microadam_kernel_times",
              "microadam_kernel_times_total", "microadam_step_noalloc"):
        getattr(lib, f).restype = ctypes.c_int
    _lib = lib
    return lib


def _check(rc: int, where: str) -> None:
    if rc != MICROADAM_OK:
        lib = load()
        raise MicroAdamError(rc, where, lib.microadam_last_error().decode() or
                             lib.microadam_error_string(rc).decode())


def make_config(density=0.01, beta1=0.9, beta2=0.999, eps=1e-8, lr=1e-4, weight_decay=0.0,
                window=10, ef_bits=4, ef_bucket=64, topk_block=4096,
                window_value_dtype=MICROADAM_BF16, ef_rounding=MICROADAM_ROUND_NEAREST,
                seed=0, fused=0) -> microadam_config:
    """A microadam_config; defaults are the paper's fine-tuning settings."""
    return microadam_config(density, beta1, beta2, eps, lr, weight_decay, window, ef_bits,
                            ef_bucket, topk_block, window_value_dtype, ef_rounding, seed, int(fused), 0)


def _i64_array(xs: Sequence[int]):
    return (ctypes.c_int64 * len(xs))(*[int(x) for x in xs])


# ---------------------------------------------------------------- C names
def microadam_state_bytes(cfg: microadam_config, numels: Sequence[int]) -> int:
    out = ctypes.c_uint64(0)
    _check(load().microadam_state_bytes(ctypes.byref(cfg), _i64_array(numels), len(numels),
                                        ctypes.byref(out)), "microadam_state_bytes")
    return out.value


def microadam_init(cfg: microadam_config, numels: Sequence[int], param_dtype: int,
                   grad_dtype: int, state_ptr: int, state_bytes: int, stream: int = 0) -> int:
    h = ctypes.c_void_p(0)
    _check(load().microadam_init(ctypes.byref(cfg), _i64_array(numels), len(numels), param_dtype,
                                 grad_dtype, ctypes.c_void_p(state_ptr), state_bytes,
                                 ctypes.c_void_p(stream), ctypes.byref(h)), "microadam_init")
    return h.value


def microadam_step(h: int, param_ptrs: Sequence[int], grad_ptrs: Sequence[int],
                   lr: float = math.nan, stream: int = 0) -> None:
    """`param_ptrs` / `grad_ptrs`: sequences of device addresses, or ctypes
    arrays of c_void_p built once and passed again (no per-call copy)."""
    n = len(param_ptrs)
    P = param_ptrs if isinstance(param_ptrs, ctypes.Array) else (ctypes.c_void_p * n)(*param_ptrs)
    G = grad_ptrs if isinstance(grad_ptrs, ctypes.Array) else (ctypes.c_void_p * len(grad_ptrs))(*grad_ptrs)
    _check(load().microadam_step(ctypes.c_void_p(h), P, G, n, float(lr), ctypes.c_void_p(stream)),
           "microadam_step")


def microadam_step_noalloc(cfg: microadam_config, numels: Sequence[int], param_dtype: int, grad_dtype: int,
                           state_ptr: int, state_bytes: int, t: int, param_ptrs: Sequence[int],
                           grad_ptrs: Sequence[int], lr: float = math.nan, stream: int = 0) -> None:
    n = len(numels)
    P = (ctypes.c_void_p * n)(*param_ptrs)
    G = (ctypes.c_void_p * n)(*grad_ptrs)
    _check(load().microadam_step_noalloc(ctypes.byref(cfg), _i64_array(numels), n, param_dtype, grad_dtype,
                                         ctypes.c_void_p(state_ptr), state_bytes, int(t), P, G, float(lr),
                                         ctypes.c_void_p(stream)), "microadam_step_noalloc")


def microadam_destroy(h: int) -> None:
    _check(load().microadam_destroy(ctypes.c_void_p(h)), "microadam_destroy")


def microadam_get_step(h: int) -> int:
    t = load().microadam_get_step(ctypes.c_void_p(h))
    if t < 0:
        _check(int(t), "microadam_get_step")
    return int(t)


def microadam_set_step(h: int, t: int) -> None:
    _check(load().microadam_set_step(ctypes.c_void_p(h), int(t)), "microadam_set_step")


def microadam_tensor_layout(h: int, tensor: int) -> microadam_layout:
    out = microadam_layout()
    _check(load().microadam_tensor_layout(ctypes.c_void_p(h), tensor, ctypes.byref(out)),
           "microadam_tensor_layout")
    return out


def microadam_debug_moments(h: int, tensor: int, mhat_ptr: int, vhat_ptr: int, stream: int = 0) -> None:
    _check(load().microadam_debug_moments(ctypes.c_void_p(h), tensor, ctypes.c_void_p(mhat_ptr),
                                          ctypes.c_void_p(vhat_ptr), ctypes.c_void_p(stream)),
           "microadam_debug_moments")


def microadam_step_kernels(h: int) -> int:
    n = load().microadam_step_kernels(ctypes.c_void_p(h))
    if n < 0:
        _check(n, "microadam_step_kernels")
    return int(n)


def microadam_set_profiling(h: int, on: bool) -> None:
    _check(load().microadam_set_profiling(ctypes.c_void_p(h), 1 if on else 0), "microadam_set_profiling")


def microadam_kernel_times(h: int) -> tuple:
    """(select ms, update ms) of the last profiled step."""
    out = (ctypes.c_float * 2)()
    _check(load().microadam_kernel_times(ctypes.c_void_p(h), out), "microadam_kernel_times")
    return float(out[0]), float(out[1])


def microadam_kernel_times_total(h: int) -> tuple:
    """(select ms, update ms, steps): durations summed over the steps profiled
    since profiling was switched on or since the previous call."""
    out = (ctypes.c_float * 2)()
    n = ctypes.c_int64()
    _check(load().microadam_kernel_times_total(ctypes.c_void_p(h), out, ctypes.byref(n)),
           "microadam_kernel_times_total")
    return float(out[0]), float(out[1]), int(n.value)


def microadam_error_string(code: int) -> str:
    return load().microadam_error_string(code).decode()


def microadam_last_error() -> str:
    return load().microadam_last_error().decode()


# ------------------------------------------------------- torch front end
class MicroAdam:
    """MicroAdam over a fixed list of CUDA(HIP) tensors.

    Allocates the optimizer state as one uint8 device tensor and drives the
    C ABI on torch's current stream.  ``step(grads)`` takes gradients of the
    same shapes; parameters are updated in place.
    """

    def __init__(self, params, cfg: microadam_config | None = None, **cfg_kw):
        import torch
        self.params = list(params)
        assert self.params, "no parameters"
        self.cfg = cfg if cfg is not None else make_config(**cfg_kw)
        dt = {torch.float32: MICROADAM_F32, torch.bfloat16: MICROADAM_BF16}
        self._dtype_code = dt
        self.param_dtype = dt[self.params[0].dtype]
        for p in self.params:
            assert p.is_cuda and p.is_contiguous() and dt[p.dtype] == self.param_dtype
        self.numels = [p.numel() for p in self.params]
        self.device = self.params[0].device
        nbytes = microadam_state_bytes(self.cfg, self.numels)
        self.state = torch.empty(nbytes + 256, dtype=torch.uint8, device=self.device)
        off = (-self.state.data_ptr()) % 256
        self.state_view = self.state[off:off + nbytes]
        self.grad_dtype = None
        self.handle = None
        # the addresses of the last checked call, and their ctypes arrays
        self._pp, self._gp = None, None
        self._parr = self._garr = None

    def _stream(self) -> int:
        import torch
        return torch.cuda.current_stream(self.device).cuda_stream

    def _ensure(self, grads) -> None:
        if self.handle is not None:
            return
        import torch
        dt = {torch.float32: MICROADAM_F32, torch.bfloat16: MICROADAM_BF16}
        self.grad_dtype = dt[grads[0].dtype]
        self.handle = microadam_init(self.cfg, self.numels, self.param_dtype, self.grad_dtype,
                                     self.state_view.data_ptr(), self.state_view.numel(),
                                     self._stream())

    def restore(self, state, t: int, grads) -> None:
        """Creates the handle for gradients like `grads`, then loads a saved
        state buffer (from ``state_view``) and step counter."""
        import torch
        self._ensure(list(grads))
        if state.numel() != self.state_view.numel():
            raise ValueError("saved state has another size")
        self.state_view.copy_(state.to(self.device, torch.uint8))
        microadam_set_step(self.handle, int(t))

    def step(self, grads, lr: float | None = None) -> None:
        grads = list(grads)
        assert len(grads) == len(self.params)
        gp = [g.data_ptr() for g in grads]
        if gp != self._gp:
            for g, p in zip(grads, self.params):
                assert g.is_contiguous() and g.numel() == p.numel() and g.device == p.device
            self._ensure(grads)
            self._garr = (ctypes.c_void_p * len(gp))(*gp)
            self._gp = gp
        else:
            # the addresses of the last checked call (so the same device);
            # the sizes are checked again
            assert [g.numel() for g in grads] == self.numels
        gdt = grads[0].dtype
        assert all(g.dtype is gdt for g in grads) and self._dtype_code.get(gdt) == self.grad_dtype, \
            "gradients of one dtype, the one of the first step"
        pp = [p.data_ptr() for p in self.params]
        if pp != self._pp:
            self._parr = (ctypes.c_void_p * len(pp))(*pp)
            self._pp = pp
        microadam_step(self.handle, self._parr, self._garr, math.nan if lr is None else lr,
                       self._stream())

    @property
    def t(self) -> int:
        return 0 if self.handle is None else microadam_get_step(self.handle)

    def layout(self, j: int) -> microadam_layout:
        return microadam_tensor_layout(self.handle, j)

    def debug_moments(self, j: int):
        import torch
        n = self.numels[j]
        m = torch.empty(n, dtype=torch.float32, device=self.device)
        v = torch.empty(n, dtype=torch.float32, device=self.device)
        microadam_debug_moments(self.handle, j, m.data_ptr(), v.data_ptr(), self._stream())
        return m, v

    @property
    def step_kernels(self) -> int:
        """Kernel launches per step: 1 (fused), 2 (select, update) or 4."""
        return microadam_step_kernels(self.handle)

    def set_profiling(self, on: bool = True) -> None:
        microadam_set_profiling(self.handle, on)

    def kernel_times(self) -> tuple:
        """(select ms, update ms) of the last step taken with profiling on."""
        return microadam_kernel_times(self.handle)

    def kernel_times_total(self) -> tuple:
        """(select ms, update ms, steps) summed over the steps profiled since
        profiling was switched on or since the previous call."""
        return microadam_kernel_times_total(self.handle)

    def close(self) -> None:
        if self.handle is not None:
            microadam_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
