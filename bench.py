#!/usr/bin/env python3
"""Throughput of the gradient sketches on one MI355X.

Workload (default): per-example gradients shaped like GPT-2 small (148
parameter tensors, N = 124,439,808 parameters), fp32 entries N(0, 1e-4),
batch 64, sketched to D = 2^16 with AFJL and with AFFD (seed 1).  One step
sketches the whole batch with both kinds; inputs are resident in HBM before
the timed region.  Prints one JSON line.

The roofline object covers the kernel class with the largest share of device
time, timed with HIP events on the stream its launches run on; its
"achieved" figure is the algorithmic bytes of those launches (inputs read
once, outputs written once) over their summed duration.  HBM traffic measured
with rocprofv3 counters is read from profiles/ when it was taken on the
current kernel source.  The fp64 oracle is timed on the host beside it on a
bounded sample.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "gradient GB/s sketched and vectors/s at N=124M, D=2^16; % HBM/MFMA peak"
HBM_PEAK_GBS = 8000.0


def gpt2_small_shapes():
    """Parameter tensors of GPT-2 small in module order (wte, wpe, 12 blocks, ln_f)."""
    s = [(50257, 768), (1024, 768)]
    for _ in range(12):
        s += [(1, 768), (1, 768),            # ln_1 weight, bias
              (768, 2304), (1, 2304),        # attn.c_attn
              (768, 768), (1, 768),          # attn.c_proj
              (1, 768), (1, 768),            # ln_2
              (768, 3072), (1, 3072),        # mlp.c_fc
              (3072, 768), (1, 768)]         # mlp.c_proj
    s += [(1, 768), (1, 768)]                # ln_f
    return s


def source_hash() -> str:
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2402_03994_amd", "csrc")
    for f in sorted(os.listdir(csrc)):
        if f.endswith((".hip", ".h")):
            h.update(open(os.path.join(csrc, f), "rb").read())
    return h.hexdigest()[:16]


def measured_traffic(kclass: str):
    """HBM bytes per algorithmic byte from a committed rocprofv3 counter summary, if current."""
    p = os.path.join(ROOT, "profiles", f"traffic_{kclass}_gpt2s_b64_d65536.json")
    if not os.path.exists(p):
        return None
    rec = json.load(open(p))
    if rec.get("source_hash") != source_hash():
        return None
    return rec


def cpu_baseline(shapes, D, seed, kinds):
    """The fp64 oracle on one batch row (all layers, every kind of the step)."""
    import numpy as np

    import oracle as O

    cores = len(os.sched_getaffinity(0))
    rng = np.random.default_rng(1002)
    xs = [(rng.standard_normal((1, r * c), dtype=np.float32) * 0.01) for r, c in shapes]
    t0 = time.perf_counter()
    for k in kinds:
        O.apply(k, shapes, D, seed, xs, nthreads=cores)
    dt = time.perf_counter() - t0
    nbytes = len(kinds) * sum(r * c for r, c in shapes) * 4
    return {"value": round(nbytes / dt / 1e9, 4), "unit": "GB/s", "cores": cores, "kind": "oracle",
            "sample": f"1 of 64 batch rows, all {len(shapes)} tensors, {'+'.join(kinds)} ({dt:.1f} s)"}


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--kinds", default="afjl,affd")
    ap.add_argument("--batch", type=int, default=64)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path (the sketch shards by "
              "batch or by layer groups with one all-reduce of [batch, D]; see DESIGN.md)", file=sys.stderr)
        return 2

    import torch

    from paper_2402_03994_amd import Sketch, _lib

    dev = torch.device("cuda", 0)
    shapes = gpt2_small_shapes()
    numels = [r * c for r, c in shapes]
    N = sum(numels)
    B, D, seed = args.batch, 1 << 16, 1
    kinds = [k for k in args.kinds.split(",") if k]

    gen = torch.Generator(device=dev).manual_seed(1002)
    xs = [torch.randn((B, n), generator=gen, device=dev, dtype=torch.float32).mul_(0.01) for n in numels]
    sks = {k: Sketch(k, shapes, D, seed, device=dev) for k in kinds}
    outs = {k: torch.empty((B, D), device=dev, dtype=torch.float32) for k in kinds}

    def step(evs=None):
        for i, k in enumerate(kinds):
            if evs is not None:
                evs[k][0].record()
            sks[k].apply(xs, out=outs[k])
            if evs is not None:
                evs[k][1].record()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()

    for k in kinds:
        sks[k].profile(True)
    per_kind = {k: 0.0 for k in kinds}
    t0 = time.perf_counter()
    for _ in range(args.steps):
        evs = {k: (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for k in kinds}
        step(evs)
        torch.cuda.synchronize()
        for k in kinds:
            per_kind[k] += evs[k][0].elapsed_time(evs[k][1])
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    prof = {k: sks[k].profile_read() for k in kinds}
    for k in kinds:
        sks[k].profile(False)

    ms = (t1 - t0) * 1e3 / args.steps
    bytes_step = len(kinds) * B * N * 4
    value = bytes_step / (ms * 1e-3) / 1e9

    # dominant kernel class by device time
    classes = {}
    for k in kinds:
        for c, (t, n, by) in prof[k].items():
            e = classes.setdefault(f"{k}:{c}", [0.0, 0, 0])
            e[0] += t
            e[1] += n
            e[2] += by
    dom = max(classes, key=lambda c: classes[c][0])
    t_dom, n_dom, by_dom = classes[dom]
    achieved = by_dom / (t_dom * 1e-3) / 1e9 if t_dom > 0 else 0.0
    tr = measured_traffic(dom.replace(":", "_"))
    roofline = {"bound": "hbm", "kernel": dom, "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                "traffic": (round(tr["hbm_bytes_per_launch"]) if tr else None),
                "launches": n_dom, "avg_launch_ms": round(t_dom / max(n_dom, 1), 4),
                "algorithmic_bytes_per_launch": round(by_dom / max(n_dom, 1))}

    line = {
        "metric": METRIC, "value": round(value, 2), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 3), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32", "data": "synthetic",
        "config": {"workload": f"GPT-2-small-shaped fp32 gradients N(0,1e-4), {len(shapes)} tensors, "
                               f"N={N}, batch {B}, D=2^16, seed 1, kinds {'+'.join(kinds)}",
                   "N": N, "batch": B, "D": D, "kinds": kinds},
        "vectors_per_s": round(B / (ms * 1e-3), 1),
        "per_kind_ms": {k: round(per_kind[k] / args.steps, 3) for k in kinds},
        "per_kind_GBps": {k: round(B * N * 4 / (per_kind[k] / args.steps * 1e-3) / 1e9, 1) for k in kinds},
        "kernel_classes_ms_per_step": {c: round(v[0] / args.steps, 3) for c, v in sorted(classes.items())},
        "roofline": roofline,
        "source_hash": source_hash(),
    }
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(shapes, D, seed, kinds)
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
