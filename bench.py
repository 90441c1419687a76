#!/usr/bin/env python3
"""MicroAdam optimizer-step benchmark on one MI355X.

Default workload: the Llama-2-7B parameter list (291 tensors, 6,738,415,616
bf16 parameters), bf16 gradients 1e-3 * Student-t(4), Top-K block 4096 at
density 1% (k = 41), window m = 10, 4-bit EF with bucket 64, lr 1e-4.

One step = one call of microadam_step over all 291 tensors: a select phase
(EF decode, block Top-K, new window row, EF re-quantisation) and an update
phase (moment rebuild from the window, parameter update).  For this workload
each phase is one kernel launch; blocks above 4096 elements run the select
phase as three launches (threshold pass, apply pass, multi-wave select of the
blocks the threshold pass left), and `--fused 1` runs the whole step as one
kernel where the configuration allows.  The W warm-up steps fill the window
(W >= m gives steady state); the K timed steps run back to back, bracketed by
device synchronisation.  Inputs are resident in HBM before timing starts: two
gradient sets are generated up front and alternate between steps.

Prints one JSON line.  `roofline` describes the dominant (longest) phase:
`achieved` is its algorithmic HBM bytes per step (fused_bytes, or
select_bytes / update_bytes) over its mean duration, timed with HIP events
that the library records on the launch stream around each phase of the timed
steps (read once after them).  `traffic` comes from the committed rocprofv3
FETCH_SIZE / WRITE_SIZE summary of that phase when it was taken on the
current kernel source, else null.  `cpu_baseline` times the CPU oracle, as it
stands, on this host's cores (one process per core, each on its own sample of
the workload's blocks) and reports the single-core rate beside it.
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
CSRC = os.path.join(ROOT, "paper_2405_15593_amd", "csrc")
# the device code: every HIP source and header of the library (the host-only
# API file excluded)
KERNEL_SOURCES = sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC)
                        if f.endswith((".hip", ".h")))
PROFILES = os.path.join(ROOT, "profiles")


def _code_only(text: str) -> str:
    """C/C++ source without comments and blank space: what the compiler sees,
    so that editing a comment does not make the stored counters stale."""
    out, i, n = [], 0, len(text)
    while i < n:
        c = text[i]
        if c in "\"'":                      # string or character literal
            j = i + 1
            while j < n and text[j] != c:
                j += 2 if text[j] == "\\" else 1
            out.append(text[i:j + 1])
            i = j + 1
        elif text.startswith("//", i):
            i = text.find("\n", i)
            i = n if i < 0 else i
        elif text.startswith("/*", i):
            i = text.find("*/", i + 2)
            i = n if i < 0 else i + 2
        else:
            out.append(c)
            i += 1
    return " ".join("".join(out).split())


def kernel_source_hash() -> str:
    """Hash of the kernel sources' code (comments and spacing excluded)."""
    h = hashlib.sha256()
    for f in KERNEL_SOURCES:
        h.update(_code_only(open(f, encoding="utf-8").read()).encode())
    return h.hexdigest()[:16]


def block_k(s: int, density: float) -> int:
    return min(s, max(1, math.ceil(density * s - 1e-9)))


def _blocks(w, n):
    nb = -(-n // w.block)
    k_total = (nb - 1) * block_k(w.block, w.density) + block_k(n - (nb - 1) * w.block, w.density)
    return nb, k_total


def select_bytes(w, ef_bits: int = 4, bucket: int | None = None) -> int:
    """Algorithmic HBM bytes of one select launch: gradient read, EF codes
    read and written (ceil(n*b/8) B each way), bucket (delta, Delta) read and
    written (8 B per bucket each way), one window row written (4 B per kept
    bf16 entry).  With buckets spanning blocks (bucket >= the block) the
    second pass reads the gradient, the codes and the new row again, and each
    block writes and the reduction reads 16 B of partials."""
    sg = w.grad_dtype.itemsize
    bucket = bucket or w.bucket
    span = bucket >= w.block and not (bucket <= 512 and w.block % bucket == 0)
    total = 0
    for n in w.numels:
        nb, k_total = _blocks(w, n)
        codes = -(-n * ef_bits // 8)
        total += n * sg + 2 * codes + 2 * 8 * (-(-n // bucket)) + 4 * k_total
        if span:
            total += n * sg + codes + 4 * k_total + 2 * 16 * nb
    return total


def update_bytes(w, t: int) -> int:
    """Algorithmic HBM bytes of one update launch at step t: parameters read
    and written, min(t, m) window rows read (4 B per bf16 entry)."""
    sp = w.param_dtype.itemsize
    rows = min(t, w.window)
    total = 0
    for n in w.numels:
        _, k_total = _blocks(w, n)
        total += 2 * n * sp + 4 * k_total * rows
    return total


def fused_bytes(w, t: int, ef_bits: int = 4) -> int:
    """Algorithmic HBM bytes of one fused step launch at step t: the select's
    bytes and the update's, less the new row's read (it stays on chip)."""
    total = select_bytes(w, ef_bits) + update_bytes(w, t)
    for n in w.numels:
        _, k_total = _blocks(w, n)
        total -= 4 * k_total
    return total


def read_traffic(kernel: str, workload: str):
    """(fetch+write bytes per launch, note) from the committed rocprofv3 summary
    of `kernel` if it matches the current kernel source, else (None, reason)."""
    path = os.path.join(PROFILES, f"traffic_{kernel}_{workload}.txt")
    if not os.path.exists(path):
        return None, f"no traffic summary {os.path.basename(path)}"
    kv = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    if kv.get("kernel_source_sha256_16") != kernel_source_hash():
        return None, "kernel changed since the counters were taken"
    try:
        return float(kv["hbm_bytes_per_launch"]), "rocprofv3 FETCH_SIZE+WRITE_SIZE, copy-calibrated"
    except (KeyError, ValueError):
        return None, "malformed traffic summary"


def _oracle_worker(args) -> tuple:
    """One CPU-baseline worker: the oracle, as it stands (single-threaded C),
    on `blocks` Top-K blocks of the workload's shape run as one tensor for
    m + 2 steps, with the workload's gradient distribution and dtypes;
    returns (parameters, seconds) of the last three steps (window full).
    Blocks are independent, so the workers' blocks are a sample of the
    workload's."""
    wname, blocks, seed = args
    import torch
    torch.set_num_threads(1)   # the input generator's threads would compete with the other workers
    import oracle
    from paper_2405_15593_amd import workloads as wl
    w = wl.WORKLOADS[wname]
    o = oracle.default()
    n = min(blocks * w.block, w.d)
    st = o.tensor(n, block=w.block, bucket=w.bucket, window=w.window, density=w.density,
                  value_bf16=True, param_bf16=w.param_dtype.itemsize == 2)
    theta = wl.draw(n, "normal", w.param_std, seed, "cpu", w.param_dtype).float().numpy()
    steps, timed_steps, timed = w.window + 2, 3, 0.0
    for t in range(1, steps + 1):
        g = wl.draw(n, w.grad_dist, w.grad_scale, wl.grad_seed(t, 0, seed), "cpu", w.grad_dtype).float().numpy()
        t0 = time.perf_counter()
        st.step(theta, g, t, w.lr)
        dt = time.perf_counter() - t0
        if t > steps - timed_steps:
            timed += dt
    return timed_steps * n, timed


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, elems_per_worker: int, workers: int) -> dict:
    """The CPU oracle on this host's cores: one worker first alone (the
    single-core rate), then `workers` at once in separate processes (started
    fresh, so they share nothing with this GPU process), each on its own
    blocks (about `elems_per_worker` parameters, at most the workload); the
    rate is all workers' parameters over the slowest worker's time."""
    import concurrent.futures as cf
    import multiprocessing as mp
    # (the budget is for the 12 steps of a window of 10; longer windows run
    # more steps on proportionally fewer parameters)
    elems = elems_per_worker * 12 // (w.window + 2)
    blocks = max(1, min(elems // w.block, -(-w.d // w.block)))
    n = min(blocks * w.block, w.d)
    ctx = mp.get_context("spawn")
    with cf.ProcessPoolExecutor(max_workers=workers, mp_context=ctx) as ex:
        n1, t1 = ex.submit(_oracle_worker, (w.name, blocks, 1000)).result()
        print(f"[bench] CPU oracle: one worker {n1 / t1:.3e} params/s", file=sys.stderr, flush=True)
        res = list(ex.map(_oracle_worker, [(w.name, blocks, 1001 + i) for i in range(workers)]))
    params = sum(r[0] for r in res)
    wall = max(r[1] for r in res)
    rate = params / wall
    dt = lambda d: "bf16" if d.itemsize == 2 else "f32"
    whole = n >= w.d
    return {"value": rate, "unit": "params/s", "cores": workers, "kind": "oracle",
            "single_core_value": n1 / t1, "nproc": os.cpu_count(), "cpu_model": cpu_model(),
            "extrapolated": not whole,
            "sample": (f"{workers} processes, each on "
                       + (f"the whole workload as one tensor of {n} params"
                          if whole else
                          f"{blocks} blocks of {w.block} ({n} params, {100.0 * n / w.d:.2f}% of the workload each)")
                       + f", {dt(w.param_dtype)} params, {dt(w.grad_dtype)} {w.grad_dist} grads, "
                       f"steps {w.window}-{w.window + 2} (window full) timed; the slowest worker took {wall:.2f} s; "
                       f"one full step {'extrapolated' if not whole else 'per process'}: {w.d / rate * workers if whole else w.d / rate:.2f} s")}


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="llama2_7b_bf16")
    ap.add_argument("--cpu-elems", type=int, default=4_096_000,
                    help="parameters per CPU-baseline worker, in whole Top-K blocks (0 disables the CPU baseline)")
    ap.add_argument("--cpu-blocks", type=int, default=None,
                    help="the same budget in Top-K blocks per worker (overrides --cpu-elems; 0 disables)")
    ap.add_argument("--cpu-workers", type=int, default=0,
                    help="CPU-baseline processes (0: the cores this process may use, at most 16)")
    ap.add_argument("--ef-bits", type=int, default=4, choices=(4, 8), help="bits per EF code")
    ap.add_argument("--ef-rounding", default="nearest", choices=("nearest", "randomized"),
                    help="EF quantizer rounding (randomized: Lemma 1)")
    ap.add_argument("--ef-bucket", type=int, default=0,
                    help="EF bucket size (0: the workload's; >= topk_block: buckets spanning blocks)")
    ap.add_argument("--fused", type=int, default=0, choices=(0, 1),
                    help="1: run each step as the one fused kernel where the configuration allows")
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
              "(the step is block-local: each GPU would step its own shard of the blocks, "
              "with no communication inside the step)",
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
    bucket = args.ef_bucket or w.bucket
    rounding = ma.MICROADAM_ROUND_RANDOMIZED if args.ef_rounding == "randomized" else ma.MICROADAM_ROUND_NEAREST
    cfg = ma.make_config(density=w.density, window=w.window, ef_bucket=bucket, topk_block=w.block, lr=w.lr,
                         ef_bits=args.ef_bits, ef_rounding=rounding, seed=1234, fused=args.fused)
    opt = ma.MicroAdam(params, cfg)

    for i in range(args.warmup):
        opt.step(grad_sets[i % 2])
    torch.cuda.synchronize()
    print(f"[bench] warm-up done (t={opt.t})", file=sys.stderr, flush=True)

    opt.set_profiling(True)
    t_first = opt.t + 1
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    for i in range(args.steps):
        opt.step(grad_sets[(args.warmup + i) % 2])
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    # the library's events around every launch of the timed steps, read once
    # after them (no synchronization between steps)
    sel_tot, upd_tot, n_timed = opt.kernel_times_total()
    assert n_timed == args.steps, (n_timed, args.steps)
    steps_t = range(t_first, t_first + args.steps)
    if opt.step_kernels == 1:
        ms = sel_tot / n_timed
        b = sum(fused_bytes(w, t, args.ef_bits) for t in steps_t) / args.steps
        kernels = {"step_kernel": {"ms": ms, "bytes": b, "gbs": b / ms / 1e6}}
    else:
        sel_ms, upd_ms = sel_tot / n_timed, upd_tot / n_timed
        sel_b = select_bytes(w, args.ef_bits, bucket)
        upd_b = sum(update_bytes(w, t) for t in steps_t) / args.steps
        large = w.block > 4096
        split = large and opt.step_kernels == 4 and not (bucket >= w.block)
        kernels = {
            "select_kernel": {"ms": sel_ms, "bytes": sel_b, "gbs": sel_b / sel_ms / 1e6,
                              "launches": (["threshold_kernel", "apply_kernel", "select_large_list_kernel"] if split
                                           else ["select_large_kernel"] if large else ["select_kernel"])},
            "update_kernel": {"ms": upd_ms, "bytes": upd_b, "gbs": upd_b / upd_ms / 1e6,
                              "launches": ["update_large_kernel" if large else "update_kernel"]},
        }
    dominant = max(kernels, key=lambda k: kernels[k]["ms"])
    dk = kernels[dominant]
    default_ef = args.ef_bits == 4 and args.ef_rounding == "nearest" and bucket == w.bucket
    traffic, traffic_note = read_traffic(dominant, w.name) if default_ef else (None, "counters taken with the default EF")
    print(f"[bench] mean kernel ms per step over {n_timed} steps: "
          f"{ {k: round(v['ms'], 3) for k, v in kernels.items()} }", file=sys.stderr, flush=True)

    cpu = None
    if args.cpu_blocks is not None:
        args.cpu_elems = args.cpu_blocks * w.block
    if args.cpu_elems > 0:
        workers = args.cpu_workers or min(16, len(os.sched_getaffinity(0)))
        print(f"[bench] CPU oracle baseline: {workers} processes x {args.cpu_elems} params", file=sys.stderr,
              flush=True)
        cpu = cpu_baseline(w, args.cpu_elems, workers)

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
            "ef_bits": args.ef_bits, "ef_rounding": args.ef_rounding, "ef_bucket": bucket,
            "steps_timed": [t_first, t_first + args.steps - 1],
            "window_full": t_first > w.window,
        },
        "kernels": kernels,
        "step_kernels": opt.step_kernels,
        "step_hbm_gbs": sum(k["bytes"] for k in kernels.values()) / sum(k["ms"] for k in kernels.values()) / 1e6,
        "roofline": {
            "bound": "hbm",
            "kernel": dominant,
            "achieved": dk["gbs"],
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": dk["gbs"] / HBM_PEAK_GBS,
            "traffic": traffic,
            "algorithmic_bytes_per_launch": dk["bytes"],
            "traffic_note": traffic_note,
        },
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)
    opt.close()
    return 0


if __name__ == "__main__":
    sys.exit(main())
