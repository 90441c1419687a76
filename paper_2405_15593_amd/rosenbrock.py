"""The two-dimensional picture behind MicroAdam's error feedback: trajectories
on the Rosenbrock function f(x, y) = (1 - x)^2 + 100 (y - x^2)^2 from
(x, y) = (-1/2, 1), as in the paper's Fig. 1 (Section 3, "Algorithm
Intuition").

Three optimizers of the figure, all binary32 torch code:

* ``adam``      Adam on the full gradient;
* ``topk``      Adam fed the Top-1 of the gradient (the larger coordinate only),
                no error feedback;
* ``topk_ef``   Adam fed the Top-1 of the accumulator a = g + e, with the
                error e = a - Top-1(a) carried to the next step (the surrogate of
                MicroAdam the figure uses);

and, on a ROCm device, MicroAdam itself through the library (``microadam``):
one 2-element tensor in a Top-K block of 16 with density 1/2, so one
coordinate is kept per step, 4-bit error feedback (a bucket of two elements
holds its min and max exactly) and a window of m sparse gradients.

    python -m paper_2405_15593_amd.rosenbrock [--steps 5000] [--lr 1e-2]
"""
from __future__ import annotations

import argparse
import json
import math

import numpy as np
import torch

START = (-0.5, 1.0)
OPTIMUM = (1.0, 1.0)


def rosenbrock(p: torch.Tensor) -> torch.Tensor:
    x, y = p[0], p[1]
    return (1 - x) ** 2 + 100 * (y - x * x) ** 2


def gradient(p: torch.Tensor) -> torch.Tensor:
    """The exact gradient of the Rosenbrock function at p (binary32)."""
    x, y = p[0], p[1]
    return torch.stack([-2 * (1 - x) - 400 * x * (y - x * x), 200 * (y - x * x)])


def _top1(v: torch.Tensor) -> torch.Tensor:
    keep = torch.zeros_like(v)
    keep[int(torch.argmax(v.abs()))] = 1
    return v * keep


def run_adam(steps: int, lr: float, compress: str = "none", device="cpu") -> np.ndarray:
    """Trajectory [steps + 1, 2] of Adam (betas 0.9, 0.999, eps 1e-8) fed the
    full gradient (``none``), its Top-1 (``topk``) or the Top-1 of the
    gradient plus the carried error (``topk_ef``)."""
    p = torch.tensor(START, dtype=torch.float32, device=device)
    p.requires_grad_(True)
    opt = torch.optim.Adam([p], lr=lr, betas=(0.9, 0.999), eps=1e-8)
    err = torch.zeros(2, dtype=torch.float32, device=device)
    traj = [p.detach().cpu().numpy().copy()]
    for _ in range(steps):
        g = gradient(p.detach())
        if compress == "topk":
            g = _top1(g)
        elif compress == "topk_ef":
            a = g + err
            g = _top1(a)
            err = a - g
        p.grad = g
        opt.step()
        traj.append(p.detach().cpu().numpy().copy())
    return np.array(traj)


def run_microadam(steps: int, lr: float, window: int = 10, device="cuda") -> np.ndarray:
    """Trajectory of MicroAdam (the library's kernels) on the 2-element
    tensor: Top-K block of 16, density 1/2 (k = 1 for the two elements),
    bucket 16, binary32 window values."""
    from . import MICROADAM_F32, MicroAdam, make_config
    p = torch.tensor(START, dtype=torch.float32, device=device)
    cfg = make_config(density=0.5, window=window, ef_bucket=16, topk_block=16, lr=lr,
                      window_value_dtype=MICROADAM_F32)
    opt = MicroAdam([p], cfg)
    traj = [p.cpu().numpy().copy()]
    try:
        for _ in range(steps):
            opt.step([gradient(p)])
            traj.append(p.cpu().numpy().copy())
    finally:
        opt.close()
    return np.array(traj)


def summary(traj: np.ndarray, reference: np.ndarray | None = None) -> dict:
    """Final point, its distance to the optimum (1, 1) and loss, the path
    length (a jagged path is long), and the largest distance from the
    reference trajectory at equal steps."""
    end = traj[-1]
    out = {
        "final": [float(end[0]), float(end[1])],
        "distance_to_optimum": float(math.hypot(end[0] - OPTIMUM[0], end[1] - OPTIMUM[1])),
        "final_loss": float(rosenbrock(torch.tensor(end, dtype=torch.float64))),
        "path_length": float(np.sum(np.hypot(*np.diff(traj, axis=0).T))),
    }
    if reference is not None:
        out["max_deviation_from_adam"] = float(np.max(np.hypot(*(traj - reference).T)))
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--steps", type=int, default=5000)
    ap.add_argument("--lr", type=float, default=1e-2)
    ap.add_argument("--window", type=int, default=10)
    ap.add_argument("--no-gpu", action="store_true", help="skip the library's MicroAdam run")
    args = ap.parse_args()
    adam = run_adam(args.steps, args.lr)
    res = {"steps": args.steps, "lr": args.lr, "start": list(START),
           "adam": summary(adam),
           "topk": summary(run_adam(args.steps, args.lr, "topk"), adam),
           "topk_ef": summary(run_adam(args.steps, args.lr, "topk_ef"), adam)}
    if not args.no_gpu and torch.cuda.is_available():
        res["microadam"] = summary(run_microadam(args.steps, args.lr, args.window), adam)
        res["microadam"]["window"] = args.window
    print(json.dumps(res))


if __name__ == "__main__":
    main()
