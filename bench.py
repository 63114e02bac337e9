#!/usr/bin/env python3
"""Throughput of the structured sketches on one MI355X.

Default workload (--config c2): per-example gradients shaped like GPT-2 small
(148 tensors, N = 124,439,808), fp32 entries N(0, 1e-4), batch 64, sketched to
D = 2^16 by AFJL and by AFFD (seed 1).  One step sketches the whole batch with
both kinds; inputs are resident in HBM before the timed region.  Other
workloads (--config c1|c3|c4|c5|c6|c7|c8|c9) are described in workloads.py; c8 times
Arnoldi on the sketched HVP operator (a step = 64 Krylov steps), c9 one whole
intrinsic-dimension search.  Prints one JSON line.

"value" is parameter-space bytes per second: gradient bytes read by forward
sketches plus parameter-vector bytes written by transposes, summed over the
calls of a step.  The roofline object covers the kernel class with the largest
share of device time among the classes that read the inputs (a class that moves
only intermediates and takes longer is named in it as largest_class), found in an
untimed calibration pass that brackets every kernel class with HIP events (the
per-class breakdown comes from it).  In the timed region only that class's
launches are bracketed, with HIP events on the stream they run on; "achieved"
is the algorithmic bytes of those launches (inputs read once, outputs written
once) over their summed duration.  "per_kind" gives the same fraction for
whole calls, every kernel of a kind included, from an untimed pass with
events around the calls only.  Traffic measured with rocprofv3 counters
(FETCH_SIZE / WRITE_SIZE: bytes between the L2 caches and the memory fabric,
so hits in the memory-side cache count too; an upper bound on HBM bytes) is
attached from profiles/ when it was taken on the current kernel source.  The
fp64 oracle is timed on the host on a bounded sample of the same workload.
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

import workloads as W  # noqa: E402

METRIC = "gradient GB/s sketched and vectors/s at N=124M, D=2^16; % HBM/MFMA peak"
HBM_PEAK_GBS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0
MFMA_F32_PEAK_TFLOPS = 157.3


# kernel launched by each single-kernel profile class (the rocprofv3 name)
KERNEL_OF = {"affd:affd_rows": "k_affdT_rows", "afjl:afjl_fold": "k_afjl_fold", "qk:qk_xb": "k_qk_s1",
             "ffd:ffd": "k_ffd_small_fwd", "ffd:gather": "k_reduce_partials", "fjl:prolog": "k_fjl_fwd_onepass",
             "afjlq:qh_first": "k_qh_gemm", "qkh:qh_first": "k_qh_gemm", "afjlq:qh_second": "k_qh_gemm",
             "qkh:qh_second": "k_qh_gemm", "affdq:qh_first": "k_qh_gemm", "affdq:qh_t": "k_qh_gemm",
             "hvp:hvp_dots": "k_hvp_dots", "hvp:hvp_combine": "k_hvp_combine", "afjl:gather": "k_afjl_T_out",
             "ffd:ffd_t": "k_ffd_small_T", "afjlf:ff_rows": "k_ffr_fwd", "afjlf:ff_small": "k_ffs_fwd",
             "afjlf:ff_res": "k_ffq_fwd", "affd:affd_fold": "k_affdT_topM", "afjl:afjl_tail": "k_afjl_tail",
             "affd:gather": "k_affdT_outm", "ffd:prolog": "k_ffd_tables",
             "fjl:fjl_t": "k_fjl_T_onepass"}
# FFD with D = 2^20 (rows / cols passes): prolog = the first rows pass of the forward, gather = the last cols
# pass of the transpose (the four-vector form when the batch is a multiple of 4); the ffd class groups the
# middle passes (several kernels)
KERNEL_OF_FFD_LARGE = {"ffd:prolog": "k_ffdL_rows<0", "ffd:gather": "k_ffdL_cols<2>",
                       "ffd:ffd": "k_ffdL middle passes"}


def kernel_of(cfg: str, kclass: str) -> str:
    c = W.CONFIGS[cfg]
    if c["D"] == 1 << 20 and kclass in KERNEL_OF_FFD_LARGE:
        if kclass == "ffd:gather" and c["batch"] % 4 == 0:
            return "k_ffdL_cols4<2>"
        return KERNEL_OF_FFD_LARGE[kclass]
    return KERNEL_OF.get(kclass, kclass)


def qk_flops(m, n, da, db):
    """MFMA flops of one vector through a QK matrix in the contraction order the library takes: A first
    (U = A X) when that makes fewer products, or when the 16-byte-load A-first kernel applies (dA <= 32,
    dA <= 2 dB, columns a multiple of 512), else B first (T = X B^T)."""
    afirst = m % 64 == 0 and n % 256 == 0 and ((da < db and da <= 64) or (da <= 32 and da <= 2 * db and n % 512 == 0))
    return 2 * da * m * n + 2 * da * n * db if afirst else 2 * m * n * db + 2 * da * m * db


def qh_flops(kind, shapes, D):
    """Multiply-add flops (2 per product) per vector of the contractions of the Q kinds, per profile
    class (qh_first reads the input, qh_second forms the output, qh_t the transpose), following the
    library's operand order."""
    first = second = trans = 0
    T, dm = 1024, D // 1024
    for r, c in shapes:
        n = r * c
        np_len = 1
        while np_len < max(n, D):
            np_len *= 2
        bm = min(1024, np_len // 1024)  # factor K - 2 (the last factor is 1024 wide)
        P = np_len // (bm * T)
        if kind == "affdq":
            for t in range(P):
                rt = min(bm, max(0, -(-(n - t * bm * T) // T)))
                first += 2 * rt * T * T + 2 * bm * rt * T
                trans += 2 * rt * bm * T + 2 * rt * T * T
            second += 2 * dm * bm * T + 2 * dm * T * T
            trans += 2 * dm * T * T + 2 * bm * dm * T
            continue
        live = -(-n // T)
        if P == 1 and live < dm:  # Qt first on the live rows, then A's live columns
            first += 2 * live * T * T
            second += 2 * dm * live * T
            trans += 2 * live * dm * T + 2 * live * T * T
        else:
            first += 2 * dm * bm * T
            second += 2 * dm * T * T
            trans += 2 * dm * T * T + 2 * bm * dm * T
    return {"qh_first": first, "qh_second": second, "qh_t": trans}


# kernel sources behind each kind (the shared headers and the dispatcher are hashed for every config)
_COMMON_SRC = ("sk_api.hip", "sk_internal.h", "sk_launch.h", "sk_kcommon.h", "sk_device.h")
_KIND_SRC = {"fjl": ("sk_fwht.hip",), "ffd": ("sk_fwht.hip", "sk_ffd_l.hip"), "afjl": ("sk_fwht.hip",),
             "affd": ("sk_fwht.hip", "sk_affd.hip", "sk_affd_s.hip", "sk_affd_t.hip"), "qk": ("sk_qk.hip",),
             "qkh": ("sk_qhaar.hip",), "afjlq": ("sk_qhaar.hip",), "affdq": ("sk_qhaar.hip",),
             "afjlf": ("sk_afjlf.hip", "sk_fft.h")}


def source_hash(cfg: str) -> str:
    """Hash of the kernel sources a workload runs: counter records taken on other sources are stale."""
    files = set(_COMMON_SRC)
    for k in W.CONFIGS[cfg]["kinds"]:
        files.update(_KIND_SRC[k])
    if cfg in ("c8", "c9"):
        files.add("sk_hvp.hip")
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2402_03994_amd", "csrc")
    for f in sorted(files):
        h.update(open(os.path.join(csrc, f), "rb").read())
    return h.hexdigest()[:16]


def measured_traffic(cfg: str, kclass: str):
    """Bytes per launch between the L2 caches and the memory fabric (rocprofv3 FETCH_SIZE + WRITE_SIZE, EA
    traffic: hits in the memory-side cache included, so an upper bound on HBM bytes) of a kernel class from a
    committed counter summary, if it was taken on the current sources."""
    p = os.path.join(ROOT, "profiles", f"traffic_{cfg}_{kclass.replace(':', '_')}.json")
    if not os.path.exists(p):
        return None
    rec = json.load(open(p))
    if rec.get("source_hash") != source_hash(cfg):
        return None
    return rec.get("ea_bytes_per_launch")


def copy_probe() -> int:
    """A plain device copy of 1 GiB, three times: the reference whose rocprofv3
    FETCH_SIZE / WRITE_SIZE readings calibrate those counters to bytes."""
    import torch

    n = (1 << 30) // 4
    src = torch.ones(n, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_bytes": n * 4, "copies": 3}), flush=True)
    return 0


def _counter_per_launch(csv_path: str, name: str, counter: str):
    import csv

    vals = {}
    for r in csv.DictReader(open(csv_path)):
        if name in r["Kernel_Name"] and r["Counter_Name"] == counter:
            vals[r["Dispatch_Id"]] = vals.get(r["Dispatch_Id"], 0.0) + float(r["Counter_Value"])
    if not vals:
        raise SystemExit(f"no {counter} records for kernels named {name!r} in {csv_path}")
    return sum(vals.values()) / len(vals), len(vals)


def traffic_json(cfg: str, kclass: str, fetch_csv: str, write_csv: str, copy_fetch_csv: str,
                 copy_write_csv: str) -> int:
    """Per-launch EA bytes (L2 <-> memory fabric) of a kernel class from rocprofv3 --pmc FETCH_SIZE and
    WRITE_SIZE runs (KiB per dispatch), each scaled by the reading for the 1 GiB
    copy of copy_probe(); written to profiles/ with the current source hash."""
    kname = kernel_of(cfg, kclass)
    f_kib, nf = _counter_per_launch(fetch_csv, kname, "FETCH_SIZE")
    w_kib, nw = _counter_per_launch(write_csv, kname, "WRITE_SIZE")
    cf_kib, _ = _counter_per_launch(copy_fetch_csv, "copy", "FETCH_SIZE")
    cw_kib, _ = _counter_per_launch(copy_write_csv, "copy", "WRITE_SIZE")
    ref_kib = (1 << 30) / 1024
    cal_f, cal_w = ref_kib / cf_kib, ref_kib / cw_kib
    rec = {"config": cfg, "class": kclass, "kernel": kname, "source_hash": source_hash(cfg),
           "fetch_kib_per_launch": round(f_kib, 1), "write_kib_per_launch": round(w_kib, 1), "launches": nf,
           "copy_fetch_kib_per_gib": round(cf_kib, 1), "copy_write_kib_per_gib": round(cw_kib, 1),
           "fetch_scale": round(cal_f, 4), "write_scale": round(cal_w, 4),
           "ea_read_bytes_per_launch": round(f_kib * 1024 * cal_f),
           "ea_write_bytes_per_launch": round(w_kib * 1024 * cal_w),
           "ea_bytes_per_launch": round(f_kib * 1024 * cal_f + w_kib * 1024 * cal_w)}
    out = os.path.join(ROOT, "profiles", f"traffic_{cfg}_{kclass.replace(':', '_')}.json")
    with open(out, "w") as fh:
        json.dump(rec, fh, indent=1)
        fh.write("\n")
    print(json.dumps(rec))
    return 0


# ------------------------------------------------------------------ CPU baseline
def cpu_baseline(cfg: str):
    """The fp64 oracle on a bounded sample of the workload (all host cores)."""
    import numpy as np

    import oracle as O

    c = W.CONFIGS[cfg]
    # the host's CPU share: OMP_NUM_THREADS where the machine sets it, else every core
    cores = int(os.environ.get("OMP_NUM_THREADS", "0") or 0) or len(os.sched_getaffinity(0))
    rng = np.random.default_rng(W.INPUT_SEED[cfg])
    shapes, D, seed = c["shapes"], c["D"], c["seed"]

    def rows_for(sh, nrows, var=1e-4):
        return [(rng.standard_normal((nrows, s[0] * s[1]), dtype=np.float32) * np.float32(np.sqrt(var)))
                for s in sh]

    t0 = None  # set in each branch once its inputs exist
    if cfg == "c1":
        xs = rows_for(shapes, c["batch"], 1.0)
        z = rng.standard_normal((c["batch"], D))
        t0 = time.perf_counter()
        reps = 0
        while reps == 0 or time.perf_counter() - t0 < 10.0:  # one pass takes well under a second
            for k in c["kinds"]:
                O.apply(k, shapes, D, seed, xs, nthreads=cores)
                O.apply_T(k, shapes, D, seed, z, nthreads=cores)
            reps += 1
        nbytes = reps * 2 * len(c["kinds"]) * c["batch"] * shapes[0][1] * 4
        sample = f"all {c['batch']} rows, FJL+FFD forward and transpose, {reps} passes"
    elif cfg in ("c2", "c10"):
        # every row of the batch over the first transformer blocks: three for the C oracle (36 tensors,
        # 21.3M parameters), two for the numpy one (24 tensors, 14.2M)
        sub, nrows = (shapes[2:38] if cfg == "c2" else shapes[2:26]), c["batch"]
        xs = rows_for(sub, nrows)
        t0 = time.perf_counter()
        for k in c["kinds"]:
            O.apply(k, sub, D, seed, xs, layer0=2, nthreads=cores)
        nbytes = len(c["kinds"]) * nrows * sum(r * cc for r, cc in sub) * 4
        names = "+".join(k.upper() for k in c["kinds"])
        sample = f"{nrows} of {c['batch']} rows, the first {len(sub) // 12} transformer blocks ({len(sub)} of " \
                 f"{len(shapes)} tensors), {names}"
    elif cfg == "c3":
        sub = shapes[1:7]  # one decoder layer: q, k, v, o, fc1, fc2
        bf = [W.bf16_bits(x) for x in rows_for(sub, 1)]
        t0 = time.perf_counter()
        O.apply("qk", sub, sum(s[2] * s[3] for s in sub), seed, bf, dtype="bf16", layer0=1, nthreads=cores)
        nbytes = sum(s[0] * s[1] for s in sub) * 2
        sample = "1 of 256 rows, one decoder layer (6 of 145 matrices), QK"
    elif cfg == "c4":
        z = rng.standard_normal((1, D))
        xs = [rng.standard_t(3, size=(1, shapes[0][1])).astype(np.float32)]
        t0 = time.perf_counter()
        O.apply_T("ffd", shapes, D, seed, z, nthreads=cores)
        O.apply("ffd", shapes, D, seed, xs, nthreads=cores)
        nbytes = 2 * shapes[0][1] * 4
        sample = "1 of 4 rows, FFD transpose and forward"
    elif cfg == "c7":
        xs = rows_for(shapes, 1, 1.0)
        z = rng.standard_normal((1, D))
        t0 = time.perf_counter()
        O.apply("affdq", shapes, D, seed, xs)
        O.apply_T("affdq", shapes, D, seed, z)
        nbytes = 2 * shapes[0][1] * 4
        sample = f"1 of {c['batch']} rows, AFFDQ forward and transpose, factor generation included"
    elif cfg == "c6":
        sub = shapes[2:14]  # one transformer block: ln_1, attn, ln_2, mlp (12 tensors)
        xs = rows_for(sub, 1)
        t0 = time.perf_counter()
        for k in c["kinds"]:
            O.apply(k, sub, D, seed, xs, layer0=2)
        nbytes = len(c["kinds"]) * sum(r * cc for r, cc in sub) * 4
        sample = f"1 of {c['batch']} rows, one transformer block (12 of {len(shapes)} tensors), AFJLQ+QKH, " \
                 "factor generation included"
    elif cfg == "c9":
        from oracle import krylov as K

        lam = np.array(W.C9_LAMBDAS, dtype=np.float32)
        hp = dict(rank=len(lam), lambdas=lam, shift=0.0, seed=W.C9_HSEED)
        v = rng.standard_normal((1, D))
        t0 = time.perf_counter()
        sub = [(1, 1 << 25)]  # the first 2^25 of the 1e8 entries: 32 of the 96 live FFD blocks
        K.sketched_hvp(c["kinds"][0], sub, D, seed, hp, v)
        nbytes = 2 * sub[0][1] * 4
        sample = "one conjugate-gradient step of the search on the first 2^25 entries: S H S^T p (FFD transpose, " \
                 "rank-8 Hessian, FFD as three fp32 parts of the fp64 HVP)"
    elif cfg == "c8":
        from oracle import krylov as K

        lam = np.array(W.C8_LAMBDAS, dtype=np.float32)
        hp = dict(rank=len(lam), lambdas=lam, shift=float(np.float32(W.C8_SHIFT)), seed=W.C8_HSEED)
        v = rng.standard_normal((1, D))
        t0 = time.perf_counter()
        K.sketched_hvp(c["kinds"][0], shapes, D, seed, hp, v)
        nbytes = 2 * sum(r * cc for r, cc in shapes) * 4
        sample = f"1 of {c['krylov']} Krylov steps: S H S^T v (AFJL transpose, rank-16 Hessian, AFJL), the " \
                 "forward sketch as three fp32 parts of the fp64 HVP"
    else:  # c5
        first, cnt = W.llama3_8b_stream_groups()[1]
        sub = shapes[first:first + cnt]
        xs = rows_for(sub, 1, 1e-5)
        bf = [W.bf16_bits(x) for x in xs]
        t0 = time.perf_counter()
        O.apply("afjl", sub, D, seed, bf, dtype="bf16", layer0=first, nthreads=cores)
        nbytes = sum(s[0] * s[1] for s in sub) * 2
        sample = "1 of 8 rows, one transformer block (9 of 291 tensors), AFJL"
    dt = time.perf_counter() - t0
    model = "unknown"
    try:
        for ln in open("/proc/cpuinfo"):
            if ln.startswith("model name"):
                model = ln.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    return {"value": round(nbytes / dt / 1e9, 4), "unit": "GB/s", "cores": cores, "kind": "oracle",
            "cpu": model, "sample": f"{sample} ({dt:.1f} s)"}


# ------------------------------------------------------------------ GPU steps
def build_step(cfg: str, dev):
    """Returns (sketches, step(evs), param_bytes_per_step, vectors_per_step, description)."""
    import torch

    from paper_2402_03994_amd import Sketch

    c = W.CONFIGS[cfg]
    shapes, D, B, seed = c["shapes"], c["D"], c["batch"], c["seed"]
    numels = [s[0] * s[1] for s in shapes]
    gen = W.generator(cfg, dev)
    bf16 = c["dtype"] == "bf16"
    dt = torch.bfloat16 if bf16 else torch.float32
    sks = {k: Sketch(k, shapes, D, seed, device=dev) for k in c["kinds"]}

    if cfg in ("c1", "c7"):
        nrot = 16  # rotate inputs so they come from HBM, not the 256 MB cache
        xs = [W.gaussian((B, numels[0]), 1.0, gen, dev) for _ in range(nrot)]
        z = torch.randn((B, D), generator=gen, device=dev)
        outs = {k: torch.empty((B, D), device=dev) for k in c["kinds"]}
        touts = {k: [torch.empty((B, numels[0]), device=dev)] for k in c["kinds"]}
        state = {"i": 0}

        def step(ev):
            x = xs[state["i"] % nrot]
            state["i"] += 1
            for k in c["kinds"]:
                ev(k, "fwd", lambda k=k: sks[k].apply([x], out=outs[k]))
                ev(k, "T", lambda k=k: sks[k].apply_T(z, outs=touts[k]))
        names = " and ".join(k.upper() for k in c["kinds"])
        return sks, step, 2 * len(c["kinds"]) * B * numels[0] * 4, B, \
            f"flat fp32 vectors N=2^20 entries N(0,1), batch {B}, D=4096, seed 0: {names} forward + transpose"

    if cfg in ("c2", "c6", "c10"):
        xs = [W.gaussian((B, n), 1e-4, gen, dev) for n in numels]
        outs = {k: torch.empty((B, D), device=dev) for k in c["kinds"]}
        sks["_inputs"] = xs

        def step(ev):
            for k in c["kinds"]:
                ev(k, "fwd", lambda k=k: sks[k].apply(xs, out=outs[k]))
        names = " and ".join(k.upper() for k in c["kinds"])
        extra = ""
        if "affd" in c["kinds"]:
            pads = [1 << max(0, (max(n, D) - 1).bit_length()) for n in numels]
            mb = sum(p for p in pads if p >= 1 << 20) * 4 / 2**20
            extra = (f"; AFFD reads the per-layer tables M = H_TT(signs . G) stored at creation "
                     f"(about {mb:.0f} MB), regenerated-Gaussian figure in affd_no_mtab")
        return sks, step, len(c["kinds"]) * B * sum(numels) * 4, B, \
            (f"GPT-2-small-shaped fp32 gradients N(0,1e-4), {len(shapes)} tensors, N={sum(numels)}, batch {B}, "
             f"D=2^16, seed 1: {names}{extra}")

    if cfg == "c3":
        # one resident input per distinct matrix shape, shared by the matrices of that shape
        bufs = {}
        for s in shapes:
            key = (s[0], s[1])
            if key not in bufs:
                bufs[key] = W.gaussian((B, s[0] * s[1]), 1e-4, gen, dev, dtype=torch.bfloat16)
        xs = [bufs[(s[0], s[1])] for s in shapes]
        out = torch.empty((B, D), device=dev)

        def step(ev):
            ev("qk", "fwd", lambda: sks["qk"].apply(xs, out=out))
        return sks, step, B * sum(numels) * 2, B, \
            (f"QK on 1.3B-decoder-shaped bf16 gradients N(0,1e-4), {len(shapes)} matrices, N={sum(numels)}, "
             f"batch {B}, D=2^18, (dA,dB) q/k/v/o 32x16, fc1 32x128, fc2 128x32, embed 256x64")

    if cfg == "c4":
        n = numels[0]
        z = torch.randn((B, D), generator=gen, device=dev)
        theta0 = W.gaussian((n,), 0.02 ** 2, gen, dev)
        theta = [torch.empty((B, n), device=dev)]
        x = W.student_t3((B, n), gen, dev)
        out = torch.empty((B, D), device=dev)

        def step(ev):
            ev("ffd", "T", lambda: sks["ffd"].apply_T(z, theta0=[theta0], outs=theta))
            ev("ffd", "fwd", lambda: sks["ffd"].apply([x], out=out))
        return sks, step, 2 * B * n * 4, B, \
            ("FFD on one 1e8-entry vector (padded to 2^27), D=2^20, batch 4: theta0 + S^T z (z ~ N(0,1)) and "
             "S x for Student-t(3) x")

    if cfg == "c9":
        from paper_2402_03994_amd import id_search

        H, _, theta0 = W.c9_problem(dev)
        work = torch.empty(int(sks[c["kinds"][0]].lib.sketch_id_search_work_floats(D)), device=dev)
        sks["hvp"] = H
        box = {}
        sks["_result"] = box

        def step(ev):
            def run():
                box["r"] = id_search(sks[c["kinds"][0]], H, theta0, c["d_min"], c["tau_target"], c["delta"],
                                     c["cg_steps"], c["max_rounds"], work=work)
            ev(c["kinds"][0], "id_search", run)
        # parameter-space bytes per sketched HVP (S^T written, S read); the count per search is known after
        # the first run (rounds x (cg_steps + 1) + the gradient at theta0)
        return sks, step, 0, 1, \
            (f"intrinsic-dimension search: FFD on a 1e8-entry vector (padded to 2^27), D_max = 2^20, quadratic "
             f"1/2 theta^T H theta with H a rank-8 synthetic Hessian, theta0 in its span; from d = {c['d_min']}, "
             f"{c['cg_steps']} CG steps per round, tau_target {c['tau_target']}, delta {c['delta']}")

    if cfg == "c8":
        from paper_2402_03994_amd import arnoldi

        H, _ = W.c8_hessian(dev)
        k = c["krylov"]
        v0 = torch.randn(D, generator=gen, device=dev)
        Q = torch.empty((k + 1, D), device=dev)
        Hb = torch.empty((k + 1, k), device=dev)
        sks["hvp"] = H
        sks["_result"] = Hb

        def step(ev):
            ev(c["kinds"][0], "arnoldi", lambda: arnoldi(sks[c["kinds"][0]], H, v0, k, Q=Q, Hbar=Hb))
        return sks, step, k * 2 * sum(numels) * 4, k, \
            (f"sketched Hessian eigenvalues: {k} Arnoldi steps (two Gram-Schmidt passes each) on v -> S H S^T v, "
             f"S = {c['kinds'][0].upper()} over GPT-2-small parameters (N={sum(numels)}), D=2^16, H = 1e-5 I + "
             f"rank-16 spike (Rademacher vectors, 14 positive and 2 negative outliers)")

    # c5
    xs = [W.gaussian((B, n), 1e-5, gen, dev, dtype=torch.bfloat16) for n in numels]
    out = torch.empty((B, D), device=dev)
    groups = W.llama3_8b_stream_groups()

    def step(ev):
        def run():
            for i, (f, cnt) in enumerate(groups):
                sks["afjl"].apply(xs[f:f + cnt], out=out, first_layer=f, accumulate=i > 0)
        ev("afjl", "fwd", run)
    return sks, step, B * sum(numels) * 2, B, \
        (f"AFJL on Llama-3-8B-shaped bf16 gradients N(0,1e-5), {len(shapes)} tensors, N={sum(numels)}, batch {B}, "
         f"D=2^20, seed 7, streamed one transformer block per call")


def call_bytes(cfg: str, kind: str, tag: str) -> int:
    """Algorithmic bytes of one call: inputs read once plus outputs written once."""
    c = W.CONFIGS[cfg]
    n = sum(s[0] * s[1] for s in c["shapes"])
    esz = 2 if c["dtype"] == "bf16" else 4
    D, B = c["D"], c["batch"]
    if tag == "fwd":
        return B * n * esz + B * D * 4
    if tag == "T":
        th = n * 4 if cfg == "c4" else 0  # theta0 read
        return B * n * 4 + B * D * 4 + th
    return 0


def per_kind_roofline(cfg: str, call_ms: dict) -> dict:
    """Whole-call figures per kind and direction: every kernel of the call counts, intermediates included."""
    out = {}
    B = W.CONFIGS[cfg]["batch"]
    for key, ms in call_ms.items():
        kind, tag = key.split(":", 1)
        by = call_bytes(cfg, kind, tag)
        if not by or not ms:
            continue
        gbs = by / (ms * 1e-3) / 1e9
        out[key] = {"ms_per_call": ms, "algorithmic_gb": round(by / 1e9, 3), "achieved_gb_s": round(gbs, 1),
                    "frac_hbm": round(gbs / HBM_PEAK_GBS, 4), "vectors_per_s": round(B / (ms * 1e-3), 1)}
    return out


def time_affd_no_mtab(xs, dev, calls: int = 5) -> dict:
    """AFFD on the same inputs with the Gaussians regenerated on every call (SK_FLAG_AFFD_NO_MTAB): no
    per-layer tables stored at creation.  Whole calls timed with HIP events after two untimed calls."""
    import torch

    from paper_2402_03994_amd import Sketch

    c = W.CONFIGS["c2"]
    sk = Sketch("affd", c["shapes"], c["D"], c["seed"], device=dev, flags=Sketch.AFFD_NO_MTAB)
    out = torch.empty((c["batch"], c["D"]), device=dev)
    for _ in range(2):
        sk.apply(xs, out=out)
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(calls):
        sk.apply(xs, out=out)
    b.record()
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / calls
    sk.close()
    by = call_bytes("c2", "affd", "fwd")
    return {"ms_per_call": round(ms, 3), "achieved_gb_s": round(by / (ms * 1e-3) / 1e9, 1),
            "frac_hbm": round(by / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            "vectors_per_s": round(c["batch"] / (ms * 1e-3), 1)}


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", default="c2", choices=sorted(W.CONFIGS))
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-probe", action="store_true", help="run the 1 GiB copy used to calibrate counters")
    ap.add_argument("--traffic-json", nargs=5, metavar=("CLASS", "FETCH_CSV", "WRITE_CSV", "COPY_FETCH_CSV",
                                                        "COPY_WRITE_CSV"),
                    help="write profiles/traffic_<config>_<class>.json from rocprofv3 counter CSVs")
    args = ap.parse_args()
    if args.copy_probe:
        return copy_probe()
    if args.traffic_json:
        return traffic_json(args.config, *args.traffic_json)
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path (the sketch shards by "
              "batch or by layer groups with one all-reduce of [batch, D])", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    dev = torch.device("cuda", 0)
    cfg = args.config
    sks, step, pbytes, vecs, desc = build_step(cfg, dev)
    result = sks.pop("_result", None)
    inputs = sks.pop("_inputs", None)
    torch.cuda.synchronize()

    def ev_none(kind, tag, fn):
        fn()

    for _ in range(args.warmup):
        step(ev_none)
    torch.cuda.synchronize()

    per_call = {}

    def ev_timed(kind, tag, fn):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        fn()
        b.record()
        per_call.setdefault(f"{kind}:{tag}", []).append((a, b))

    # call timing pass (untimed): HIP events around every call only
    ncal = max(1, min(args.steps, 3))
    for _ in range(ncal):
        step(ev_timed)
    torch.cuda.synchronize()
    call_ms = {k: round(sum(a.elapsed_time(b) for a, b in v) / ncal, 3) for k, v in per_call.items()}

    # calibration pass (untimed): HIP events around every kernel-class launch
    # group, to find the class with the largest share of device time and to
    # report the per-class breakdown
    for s in sks.values():
        s.profile(True)
    for _ in range(ncal):
        step(ev_none)
    torch.cuda.synchronize()
    cal = {k: s.profile_read() for k, s in sks.items()}
    for s in sks.values():
        s.profile(False)
    classes = {}
    for k in sks:
        for cl, (t, n, by) in cal[k].items():
            e = classes.setdefault(f"{k}:{cl}", [0.0, 0, 0])
            e[0] += t
            e[1] += n
            e[2] += by
    # the dominant kernel class: the largest by device time among the classes that read the inputs (their
    # algorithmic bytes give "achieved"); when a class that moves only intermediates takes more time, it is
    # named beside it (largest_class), and per_kind covers every kernel of each call
    dom_any = max(classes, key=lambda c: classes[c][0])
    cands = [c for c in classes if classes[c][2] > 0] or list(classes)
    dom = max(cands, key=lambda c: classes[c][0])
    dom_kind, dom_cls = dom.split(":", 1)

    # timed region: K steps, with HIP events (on the stream the kernels run on)
    # around the launches of the dominant class only
    sks[dom_kind].profile(True, classes=[dom_cls])
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step(ev_none)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    t_dom, n_dom, by_dom = sks[dom_kind].profile_read()[dom_cls]
    sks[dom_kind].profile(False)

    ms = (t1 - t0) * 1e3 / args.steps
    if cfg == "c9":
        r = result["r"]
        c = W.CONFIGS[cfg]
        hvps = r["rounds"] * (c["cg_steps"] + 1)  # the sketched HVPs of the search (+ the gradient at theta0)
        pbytes = (2 * hvps + 1) * c["shapes"][0][0] * c["shapes"][0][1] * 4
    value = pbytes / (ms * 1e-3) / 1e9
    achieved = by_dom / (t_dom * 1e-3) / 1e9 if t_dom > 0 else 0.0
    roofline = {"bound": "hbm", "kernel": kernel_of(cfg, dom), "class": dom, "achieved": round(achieved, 1),
                "peak": HBM_PEAK_GBS,
                "unit": "GB/s", "frac": round(achieved / HBM_PEAK_GBS, 4),
                "traffic": measured_traffic(cfg, dom),
                "launches": n_dom, "avg_launch_ms": round(t_dom / max(n_dom, 1), 4),
                "algorithmic_bytes_per_launch": round(by_dom / max(n_dom, 1))}
    if dom_any != dom:
        roofline["largest_class"] = {"class": dom_any, "kernel": kernel_of(cfg, dom_any),
                                     "ms_per_step": round(classes[dom_any][0] / ncal, 3),
                                     "reads": "intermediates only (no algorithmic bytes)"}
    if cfg == "c3":
        c = W.CONFIGS[cfg]
        flops = sum(qk_flops(*s) for s in c["shapes"]) * c["batch"]
        roofline["mfma_tflops"] = round(flops / (t_dom * 1e-3 / args.steps) / 1e12, 1)
        roofline["mfma_frac"] = round(roofline["mfma_tflops"] / MFMA_BF16_PEAK_TFLOPS, 4)
    if cfg in ("c6", "c7"):
        # fp32 MFMA contractions: the bound is the larger of the two fractions
        c = W.CONFIGS[cfg]
        flops = qh_flops(dom_kind, c["shapes"], c["D"])[dom_cls] * c["batch"] * args.steps
        tf = flops / (t_dom * 1e-3) / 1e12 if t_dom > 0 else 0.0
        roofline["mfma_tflops"] = round(tf, 1)
        roofline["mfma_frac"] = round(tf / MFMA_F32_PEAK_TFLOPS, 4)
        roofline["flops_per_launch"] = round(flops / max(n_dom, 1))
        if tf / MFMA_F32_PEAK_TFLOPS > roofline["frac"]:
            roofline.update({"bound": "mfma", "achieved": round(tf, 1), "peak": MFMA_F32_PEAK_TFLOPS,
                             "unit": "TFLOP/s", "frac": round(tf / MFMA_F32_PEAK_TFLOPS, 4)})

    line = {
        "metric": METRIC, "value": round(value, 2), "unit": "GB/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 3), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": W.CONFIGS[cfg]["dtype"], "data": "synthetic",
        "config": {"workload": desc, "name": cfg, "batch": W.CONFIGS[cfg]["batch"], "D": W.CONFIGS[cfg]["D"],
                   "kinds": list(W.CONFIGS[cfg]["kinds"])},
        "vectors_per_s": round(vecs / (ms * 1e-3), 1),
        "per_call_ms": call_ms,
        "per_kind": per_kind_roofline(cfg, call_ms),
        "kernel_classes_ms_per_step": {c: round(v[0] / ncal, 3) for c, v in sorted(classes.items())},
        "roofline": roofline,
        "source_hash": source_hash(cfg),
    }
    if cfg == "c9":
        r = result["r"]
        line.pop("vectors_per_s")
        line["searches_per_s"] = round(1e3 / ms, 2)
        line["search"] = {"d": r["d"], "status": r["status"], "rounds": r["rounds"], "ds": r["ds"],
                          "taus": [round(t, 4) for t in r["taus"]]}
    if cfg == "c8":
        from paper_2402_03994_amd import ritz_values

        ritz = np.sort(ritz_values(result).real)[::-1]
        line["config"]["krylov"] = W.CONFIGS[cfg]["krylov"]
        line["krylov_steps_per_s"] = line.pop("vectors_per_s")
        line["ritz_top"] = [round(float(v), 4) for v in ritz[:6]] + [round(float(v), 4) for v in ritz[-2:]]
        line["hessian_spikes"] = sorted(W.C8_LAMBDAS, reverse=True)
    if cfg == "c2" and inputs is not None:
        line["affd_no_mtab"] = time_affd_no_mtab(inputs, dev)
    if not args.no_cpu_baseline:
        line["cpu_baseline"] = cpu_baseline(cfg)
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
