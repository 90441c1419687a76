"""Seeded synthetic workloads: parameter-list shapes of the models the MicroAdam
paper fine-tunes (BERT-base, Llama-2-7B/13B) and flat tensors, with the
hyper-parameters the paper trains with (Appendix B).  Gradients and initial
parameters are generated on the device with torch generators.

This module holds no arithmetic of the method: it only draws inputs, which
the HIP path and the oracle then both consume bit for bit.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import torch


def bert_base_shapes() -> list[tuple[int, ...]]:
    """196 tensors, 108,890,112 parameters: word (30522x768) and position
    (512x768) embeddings, the embedding LayerNorm, and 12 encoder layers of
    Q/K/V/O 768x768 with biases, FFN 768x3072 / 3072x768 with biases and two
    LayerNorms (gamma, beta)."""
    h, f = 768, 3072
    shapes: list[tuple[int, ...]] = [(30522, h), (512, h), (h,), (h,)]
    for _ in range(12):
        for _ in range(4):
            shapes += [(h, h), (h,)]
        shapes += [(h, f), (f,), (f, h), (h,)]
        shapes += [(h,), (h,), (h,), (h,)]
    return shapes


def llama2_shapes(hidden: int, inter: int, layers: int, vocab: int = 32000) -> list[tuple[int, ...]]:
    """Embedding, per layer Q/K/V/O (hidden^2), gate/up (hidden x inter), down
    (inter x hidden) and two RMSNorm vectors, the final norm and the LM head."""
    shapes: list[tuple[int, ...]] = [(vocab, hidden)]
    for _ in range(layers):
        shapes += [(hidden, hidden)] * 4
        shapes += [(inter, hidden), (inter, hidden), (hidden, inter)]
        shapes += [(hidden,), (hidden,)]
    shapes += [(hidden,), (vocab, hidden)]
    return shapes


@dataclass
class Workload:
    name: str
    shapes: list[tuple[int, ...]]
    param_dtype: torch.dtype
    grad_dtype: torch.dtype
    grad_dist: str              # a distribution name of draw()
    grad_scale: float
    block: int = 4096
    density: float = 0.01
    window: int = 10
    bucket: int = 64
    lr: float = 1e-4
    steps: int = 5
    param_std: float = 0.02
    notes: str = ""
    numels: list[int] = field(init=False)

    def __post_init__(self):
        self.numels = [int(torch.Size(s).numel()) for s in self.shapes]

    @property
    def d(self) -> int:
        return sum(self.numels)


WORKLOADS = {
    "flat1m_f32": Workload("flat1m_f32", [(1_048_576,)], torch.float32, torch.float32,
                           "normal", 1.0, steps=20,
                           notes="one flat tensor; grads N(0,1) fresh each step"),
    "bert_base_bf16": Workload("bert_base_bf16", bert_base_shapes(), torch.bfloat16,
                               torch.bfloat16, "normal", 1e-3, steps=10),
    "llama2_7b_bf16": Workload("llama2_7b_bf16", llama2_shapes(4096, 11008, 32),
                               torch.bfloat16, torch.bfloat16, "student_t4", 1e-3, steps=5),
    "llama2_13b_bf16": Workload("llama2_13b_bf16", llama2_shapes(5120, 13824, 40),
                                torch.bfloat16, torch.bfloat16, "normal", 1e-3, steps=3),
    "flat1p5b_ties_bf16": Workload("flat1p5b_ties_bf16", [(1_500_000_000,)], torch.bfloat16,
                                   torch.bfloat16, "student_t2_snapped64", 1e-3, block=65536,
                                   density=0.05, window=20, bucket=128, steps=5),
}


def grad_seed(step: int, tensor: int, base: int = 0) -> int:
    """Seed of the gradient of `tensor` at step `step` (1-based)."""
    return base + 1_000_003 * step + tensor


def _gen(device, seed: int) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return g


def draw(n: int, dist: str, scale: float, seed: int, device, dtype) -> torch.Tensor:
    """n values of the named distribution, times `scale`, rounded to dtype."""
    g = _gen(device, seed)
    z = torch.randn(n, generator=g, device=device, dtype=torch.float32)
    if dist == "normal":
        x = z
    elif dist in ("student_t4", "student_t2", "student_t2_snapped64"):
        df = 4 if dist == "student_t4" else 2
        chi2 = torch.zeros(n, device=device, dtype=torch.float32)
        for _ in range(df):   # chi-square with df degrees: sum of df squared normals
            w = torch.randn(n, generator=g, device=device, dtype=torch.float32)
            chi2.add_(w * w)
        x = z / torch.sqrt(chi2 / df)
        if dist == "student_t2_snapped64":
            # keep the sign, snap |x * scale| to the nearest (in log2) of the 64
            # levels scale * 2^((j - 40) / 4), j = 0..63 (lower j on a tie,
            # clamped at both ends): thousands of exact ties per block.
            j = torch.round(torch.log2(x.abs().clamp_min(1e-30)) * 4 + 40 - 1e-6)
            j = j.clamp(0, 63)
            x = torch.sign(x) * torch.exp2((j - 40) / 4)
            x = torch.where(x == 0, torch.exp2(torch.tensor(-10.0, device=device)), x)
    elif dist == "zeros":
        x = torch.zeros_like(z)
    elif dist == "constant":
        x = torch.ones_like(z)
    elif dist == "signs":          # +1 or -1: every |x| ties
        x = torch.where(z < 0, -1.0, 1.0)
    elif dist == "sparse_spikes":  # about 1 in 200 elements nonzero, the rest exact zeros
        x = torch.where(z.abs() > 2.807, z, torch.zeros_like(z))
    else:
        raise ValueError(dist)
    return (x * scale).to(dtype)


def init_params(w: Workload, device, seed: int = 0) -> list[torch.Tensor]:
    """theta_0 ~ N(0, param_std) per tensor, seeded per tensor."""
    return [draw(n, "normal", w.param_std, seed + 7919 * (j + 1), device, w.param_dtype)
            for j, n in enumerate(w.numels)]


def grads_for_step(w: Workload, step: int, device, seed_base: int = 0) -> list[torch.Tensor]:
    return [draw(n, w.grad_dist, w.grad_scale, grad_seed(step, j, seed_base), device, w.grad_dtype)
            for j, n in enumerate(w.numels)]


def grad_for_tensor(w: Workload, step: int, j: int, device, seed_base: int = 0) -> torch.Tensor:
    return draw(w.numels[j], w.grad_dist, w.grad_scale, grad_seed(step, j, seed_base), device,
                w.grad_dtype)
