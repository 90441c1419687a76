#!/usr/bin/env python3
"""MicroAdam optimizer-step benchmark on one MI355X.

Default workload: the Llama-2-7B parameter list (291 tensors, 6,738,415,616
bf16 parameters), bf16 gradients 1e-3 * Student-t(4), Top-K block 4096 at
density 1% (k = 41), window m = 10, 4-bit EF with bucket 64, lr 1e-4.

One step = one call of microadam_step over all 291 tensors (one kernel
launch).  The W warm-up steps fill the window (W >= m gives steady state);
the K timed steps run back to back, bracketed by device synchronisation.
Inputs are resident in HBM before timing starts: two gradient sets are
generated up front and alternate between steps.

Prints one JSON line.  `roofline.achieved` is the algorithmic HBM bytes of
one launch (see step_bytes) over the mean kernel duration, timed with HIP
events on the launch stream.  `roofline.traffic` comes from the committed
rocprofv3 FETCH_SIZE / WRITE_SIZE summary when it was taken on the current
kernel source, else null.  `cpu_baseline` times the CPU oracle on a sample
of the same workload's blocks on this host.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "MicroAdam step params/sec + achieved HBM GB/s (% peak), Llama-2-7B shape"
HBM_PEAK_GBS = 8000.0
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2405_15593_amd", "csrc", f)
                  for f in ("microadam_kernels.hip", "microadam_device.h")]
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic_step_kernel_llama2_7b_bf16.txt")


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        h.update(open(f, "rb").read())
    return h.hexdigest()[:16]


def block_k(s: int, density: float) -> int:
    return min(s, max(1, math.ceil(density * s - 1e-9)))


def step_bytes(w, t: int) -> int:
    """Algorithmic HBM bytes of step t: gradient read, parameter read and
    write, EF codes read and write (ceil(n/2) B), bucket (delta, Delta) read and
    write (8 B per bucket), one window row written and min(t, m) - 1 older rows
    read (4 B per bf16 entry)."""
    sg = w.grad_dtype.itemsize
    sp = w.param_dtype.itemsize
    rows_read = min(t, w.window) - 1
    total = 0
    for n in w.numels:
        nb = -(-n // w.block)
        k_total = (nb - 1) * block_k(w.block, w.density) + block_k(n - (nb - 1) * w.block, w.density)
        total += n * sg + 2 * n * sp + 2 * ((n + 1) // 2) + 2 * 8 * (-(-n // w.bucket))
        total += 4 * k_total * (1 + rows_read)
    return total


def read_traffic():
    """(fetch+write bytes per launch, note) from the committed rocprofv3 summary
    if it matches the current kernel source, else (None, reason)."""
    if not os.path.exists(TRAFFIC_FILE):
        return None, "no traffic summary"
    kv = {}
    for line in open(TRAFFIC_FILE):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    if kv.get("kernel_source_sha256_16") != kernel_source_hash():
        return None, "kernel changed since the counters were taken"
    try:
        return float(kv["hbm_bytes_per_launch"]), "rocprofv3 FETCH_SIZE+WRITE_SIZE, copy-calibrated"
    except (KeyError, ValueError):
        return None, "malformed traffic summary"


def cpu_baseline(w, blocks: int, seed: int = 0) -> dict:
    """The CPU oracle (single-threaded, as it stands) on `blocks` Top-K blocks
    of the workload's shape, run to steady state (m + 2 steps); the last two
    steps are timed."""
    import numpy as np
    import oracle
    o = oracle.default()
    n = blocks * w.block
    st = o.tensor(n, block=w.block, bucket=w.bucket, window=w.window, density=w.density,
                  value_bf16=True, param_bf16=True)
    rng = np.random.default_rng(seed)
    theta = (rng.standard_normal(n) * w.param_std).astype(np.float32)
    import torch
    theta = torch.from_numpy(theta).to(torch.bfloat16).float().numpy()
    timed = 0.0
    steps = w.window + 2
    for t in range(1, steps + 1):
        g = (rng.standard_t(4, n) * w.grad_scale).astype(np.float32)
        g = torch.from_numpy(g).to(torch.bfloat16).float().numpy()
        t0 = time.perf_counter()
        st.step(theta, g, t, w.lr)
        dt = time.perf_counter() - t0
        if t > steps - 2:
            timed += dt
    rate = 2 * n / timed
    return {"value": rate, "unit": "params/s", "cores": 1, "kind": "oracle",
            "sample": (f"{blocks} blocks of {w.block} ({n} params), bf16, steps {steps - 1}-{steps} "
                       f"(window full) timed, {timed:.2f} s")}


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="llama2_7b_bf16")
    ap.add_argument("--cpu-blocks", type=int, default=4000, help="0 disables the CPU baseline")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run a plain 4 GiB device-to-device copy three times (the known-size "
                         "kernel that scales rocprofv3 FETCH_SIZE / WRITE_SIZE to bytes)")
    args = ap.parse_args()
    if args.copy_calibration:
        import torch
        src = torch.ones(1 << 31, dtype=torch.bfloat16, device="cuda:0")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": src.numel() * 2, "copy_bytes_written": dst.numel() * 2}))
        return 0
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported "
              "(the MicroAdam step needs no communication; see DESIGN.md for sharding)",
              file=sys.stderr)
        return 2

    import torch
    import paper_2405_15593_amd as ma
    from paper_2405_15593_amd import workloads as wl

    ma.load()  # fails loudly when the HIP library is missing
    w = wl.WORKLOADS[args.workload]
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    print(f"[bench] {w.name}: {len(w.numels)} tensors, d={w.d}", file=sys.stderr, flush=True)
    params = wl.init_params(w, dev, seed=0)
    grad_sets = [wl.grads_for_step(w, s, dev) for s in (1, 2)]
    torch.cuda.synchronize()
    print("[bench] inputs resident", file=sys.stderr, flush=True)
    cfg = ma.make_config(density=w.density, window=w.window, ef_bucket=w.bucket,
                         topk_block=w.block, lr=w.lr)
    opt = ma.MicroAdam(params, cfg)
    stream = torch.cuda.current_stream(dev)

    for i in range(args.warmup):
        opt.step(grad_sets[i % 2])
    torch.cuda.synchronize()
    print(f"[bench] warm-up done (t={opt.t})", file=sys.stderr, flush=True)

    starts = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    ends = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    t_first = opt.t + 1
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    for i in range(args.steps):
        starts[i].record(stream)
        opt.step(grad_sets[(args.warmup + i) % 2])
        ends[i].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    kernel_ms = [s.elapsed_time(e) for s, e in zip(starts, ends)]
    mean_kernel_s = sum(kernel_ms) / len(kernel_ms) / 1e3
    nbytes = [step_bytes(w, t) for t in range(t_first, t_first + args.steps)]
    bytes_per_launch = sum(nbytes) / len(nbytes)
    achieved = bytes_per_launch / mean_kernel_s / 1e9
    traffic, traffic_note = read_traffic()
    print(f"[bench] kernel ms per step: {[round(x, 3) for x in kernel_ms]}", file=sys.stderr, flush=True)

    cpu = None
    if args.cpu_blocks > 0:
        print(f"[bench] CPU oracle baseline on {args.cpu_blocks} blocks", file=sys.stderr, flush=True)
        cpu = cpu_baseline(w, args.cpu_blocks)

    ms_per_step = wall / args.steps * 1e3
    out = {
        "metric": METRIC,
        "value": w.d * args.steps / wall,
        "unit": "params/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "config": {
            "workload": w.name, "params": w.d, "tensors": len(w.numels),
            "param_dtype": "bf16" if w.param_dtype.itemsize == 2 else "f32",
            "grad_dtype": "bf16" if w.grad_dtype.itemsize == 2 else "f32",
            "grad_dist": w.grad_dist, "topk_block": w.block, "density": w.density,
            "k_per_block": block_k(w.block, w.density), "window": w.window,
            "ef_bits": 4, "ef_bucket": w.bucket, "steps_timed": [t_first, t_first + args.steps - 1],
            "window_full": t_first > w.window,
        },
        "kernel_ms_mean": mean_kernel_s * 1e3,
        "hbm_gbs": achieved,
        "roofline": {
            "bound": "hbm",
            "achieved": achieved,
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS,
            "traffic": traffic,
            "algorithmic_bytes_per_launch": bytes_per_launch,
            "traffic_note": traffic_note,
        },
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)
    opt.close()
    return 0


if __name__ == "__main__":
    sys.exit(main())
