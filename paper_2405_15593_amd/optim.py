"""``torch.optim`` front-end over the C ABI: MicroAdam (Algorithm 1) with
decoupled weight decay (Algorithm 4).

Each parameter group is stepped by one library handle per parameter dtype
(the C ABI takes one parameter dtype and one gradient dtype per handle).  The
group's ``lr`` is passed at every step, so learning-rate schedulers work; the
other hyper-parameters of a group are fixed when its handle is created, at the
group's first step.  Every step of the method runs in the library's kernels;
this module only groups tensors and hands over pointers.
"""
from __future__ import annotations

import torch

from . import MICROADAM_BF16, MICROADAM_F32, MicroAdam, make_config

_DTYPES = {torch.float32: MICROADAM_F32, torch.bfloat16: MICROADAM_BF16}


class MicroAdamW(torch.optim.Optimizer):
    """MicroAdam for parameters on a ROCm device (float32 or bfloat16,
    contiguous).  Defaults are the paper's fine-tuning settings (Appendix B):
    density 1% per Top-K block of 4096, a window of m = 10 rows, 4-bit error
    feedback in buckets of 64, no weight decay."""

    def __init__(self, params, lr: float = 1e-4, betas=(0.9, 0.999), eps: float = 1e-8,
                 weight_decay: float = 0.0, density: float = 0.01, window: int = 10,
                 ef_bucket: int = 64, topk_block: int = 4096, window_values: str = "bf16"):
        if not lr >= 0.0:
            raise ValueError(f"invalid lr {lr}")
        if not (0.0 <= betas[0] < 1.0 and 0.0 <= betas[1] < 1.0):
            raise ValueError(f"invalid betas {betas}")
        if not eps >= 0.0:
            raise ValueError(f"invalid eps {eps}")
        if not weight_decay >= 0.0:
            raise ValueError(f"invalid weight_decay {weight_decay}")
        if not 0.0 < density <= 1.0:
            raise ValueError(f"invalid density {density}")
        if window_values not in ("bf16", "f32"):
            raise ValueError("window_values must be 'bf16' or 'f32'")
        defaults = dict(lr=lr, betas=tuple(betas), eps=eps, weight_decay=weight_decay,
                        density=density, window=window, ef_bucket=ef_bucket,
                        topk_block=topk_block, window_values=window_values)
        super().__init__(params, defaults)
        self._engines: dict = {}   # (group index, dtype) -> MicroAdam
        self._restore: dict = {}   # saved engine states waiting for their first step

    # ------------------------------------------------------------- engines
    @staticmethod
    def _key(gi: int, dtype: torch.dtype) -> str:
        return f"{gi}:{str(dtype).replace('torch.', '')}"

    def _engine(self, gi: int, group: dict, params: list, grads: list) -> MicroAdam:
        key = self._key(gi, params[0].dtype)
        eng = self._engines.get(key)
        if eng is None:
            cfg = make_config(density=group["density"], beta1=group["betas"][0],
                              beta2=group["betas"][1], eps=group["eps"], lr=group["lr"],
                              weight_decay=group["weight_decay"], window=group["window"],
                              ef_bucket=group["ef_bucket"], topk_block=group["topk_block"],
                              window_value_dtype=(MICROADAM_F32 if group["window_values"] == "f32"
                                                  else MICROADAM_BF16))
            eng = MicroAdam(params, cfg)
            saved = self._restore.pop(key, None)
            if saved is not None:
                eng.restore(saved["state"], int(saved["t"]), grads)
            self._engines[key] = eng
        return eng

    def state_bytes(self) -> int:
        """Bytes of device state held by the handles created so far."""
        return sum(int(e.state.numel()) for e in self._engines.values())

    # ---------------------------------------------------------------- step
    @torch.no_grad()
    def step(self, closure=None):
        loss = None
        if closure is not None:
            with torch.enable_grad():
                loss = closure()
        for gi, group in enumerate(self.param_groups):
            by_dtype: dict = {}
            for p in group["params"]:
                if p.dtype not in _DTYPES:
                    raise TypeError(f"MicroAdamW supports float32 and bfloat16 parameters, not {p.dtype}")
                by_dtype.setdefault(p.dtype, []).append(p)
            for ps in by_dtype.values():
                if all(p.grad is None for p in ps):
                    continue
                # a parameter without a gradient takes a zero gradient; one
                # gradient dtype per handle (that of the first gradient)
                gdt = next(p.grad.dtype for p in ps if p.grad is not None)
                grads = []
                for p in ps:
                    g = p.grad if p.grad is not None else torch.zeros_like(p, dtype=gdt)
                    if g.dtype != gdt:
                        g = g.to(gdt)
                    grads.append(g.contiguous())
                self._engine(gi, group, ps, grads).step(grads, lr=group["lr"])
        return loss

    # ------------------------------------------------------- checkpointing
    def state_dict(self):
        sd = super().state_dict()
        sd["microadam"] = {k: {"t": e.t, "state": e.state_view.detach().clone()}
                           for k, e in self._engines.items()}
        return sd

    def load_state_dict(self, state_dict):
        state_dict = dict(state_dict)
        saved = state_dict.pop("microadam", {})
        super().load_state_dict(state_dict)
        self._engines.clear()
        self._restore = {k: v for k, v in saved.items()}
