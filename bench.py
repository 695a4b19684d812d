#!/usr/bin/env python3
"""Throughput of the spectral spin-weighted spherical convolution layer on one
MI355X: spin_sph_conv_forward on a 256 x 256 grid, bandlimit 128, batch 2,
spins {0,1} -> {0,1}, 256 -> 256 channels, bfloat16 storage with float32
accumulation (the large weather-shaped workload).

    python bench.py [--steps K] [--warmup W] [--gpus 1] [--no-cpu-baseline]
    python bench.py --summarize-counters FETCH_CSV WRITE_CSV

Prints one JSON line.  A step is one layer call (forward transform, per-degree
mixing, inverse transform) on inputs resident in HBM.  `value` is layer calls
per second over the K timed steps.  The roofline object describes the stage
that takes the most time, measured with HIP events recorded around each of
its launches on the stream it runs on, over a second pass of K steps.  The
cpu_baseline object times the float64 oracle on the host cores on the same
workload (three layer calls, median).
"""

from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0
PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}   # dense MFMA, MI355X datasheet
METRIC = "spin-sph-conv layer fwd/sec + TFLOP/s & % MFMA peak at 256² grid, C=256"


def stage_work(w):
    """Algorithmic flops and bytes of each stage of one layer call.

    Flops count only the contractions that the layer needs: triangular
    degree ranges (l >= max(|m|, |s|)) and spins that exist at a degree.
    Bytes count one read of every operand and one write of every result in
    the storage type; X and Y are the longitude spectra between the DFT and
    latitude stages, S (2L-1) B C H complex values.
    """
    e = 2 if w.dtype == "bf16" else 4
    H, W, L, B = w.H, w.W, w.L, w.B
    Si, So, Ci, Co = len(w.spins_in), len(w.spins_out), w.C_in, w.C_out
    M = 2 * L - 1
    x_b = B * Si * Ci * H * W * 2 * e
    y_b = B * So * Co * H * W * 2 * e
    X_b = Si * M * B * Ci * H * 2 * e
    Y_b = So * M * B * Co * H * 2 * e
    a_b = L * L * B * Si * Ci * 2 * e
    a2_b = L * L * B * So * Co * 2 * e
    K_b = L * So * Co * Si * Ci * 2 * e
    tab_i = sum(sum(L - max(abs(m), abs(s)) for m in range(-(L - 1), L)) for s in w.spins_in) * H * e
    tab_o = sum(sum(L - max(abs(m), abs(s)) for m in range(-(L - 1), L)) for s in w.spins_out) * H * e
    lat_f = sum(4 * H * B * Ci * (L * L - s * s) for s in w.spins_in)
    lat_i = sum(4 * H * B * Co * (L * L - s * s) for s in w.spins_out)
    mix = 0
    for l in range(L):
        k = Ci * sum(1 for s in w.spins_in if abs(s) <= l)
        n = Co * sum(1 for t in w.spins_out if abs(t) <= l)
        mix += 8 * B * (2 * l + 1) * k * n
    return {
        "dft_fwd": {"flops": 0, "bytes": x_b + X_b},
        "lat_fwd": {"flops": lat_f, "bytes": X_b + tab_i + a_b},
        "mix": {"flops": mix, "bytes": a_b + K_b + a2_b},
        "lat_inv": {"flops": lat_i, "bytes": a2_b + tab_o + Y_b},
        "dft_inv": {"flops": 0, "bytes": Y_b + y_b},
    }


def source_digest() -> str:
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2306_05420_amd", "csrc")
    for name in sorted(os.listdir(csrc)):
        with open(os.path.join(csrc, name), "rb") as f:
            h.update(name.encode() + f.read())
    return h.hexdigest()[:16]


def measured_traffic(kernel: str):
    """HBM bytes per launch from the committed counter summary, if it was
    taken on the current kernel sources (else None)."""
    path = os.path.join(ROOT, "profiles", "traffic_wx256.json")
    try:
        with open(path) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("source_digest") != source_digest():
        return None
    k = rec.get("kernels", {}).get(kernel)
    return None if k is None else k.get("hbm_bytes_per_launch")


STAGE_KERNELS = re.compile(r"(dft_fwd|dft_inv|lat_fwd|lat_inv|mix)(?:_dma)?_kernel")
COPY_KERNEL = "__amd_rocclr_copyBuffer"
COPY_BYTES = 1 << 30


def summarize_counters(fetch_csv: str, write_csv: str, out_path: str) -> dict:
    """HBM bytes per launch of each stage kernel from two rocprofv3 counter
    runs of this script (FETCH_SIZE, then WRITE_SIZE, both with
    --copy-calibration).  Each counter (KiB per dispatch) is scaled by what it
    reads for the plain 1 GiB device copy in the same run; the median over a
    kernel's dispatches is kept."""
    import csv
    import statistics

    def per_kernel(path, counter):
        vals, copies = {}, []
        with open(path) as f:
            for r in csv.DictReader(f):
                if r["Counter_Name"] != counter:
                    continue
                v = float(r["Counter_Value"]) * 1024.0
                if r["Kernel_Name"].startswith(COPY_KERNEL):
                    copies.append(v)
                    continue
                m = STAGE_KERNELS.search(r["Kernel_Name"])
                if m:
                    vals.setdefault(m.group(1), []).append(v)
        if not copies:
            raise SystemExit(f"{path}: no {COPY_KERNEL} dispatch (run with --copy-calibration)")
        scale = COPY_BYTES / max(copies)  # the 1 GiB copy is the largest one
        return {k: statistics.median(v) for k, v in vals.items()}, scale, len(copies)

    fetch, f_scale, _ = per_kernel(fetch_csv, "FETCH_SIZE")
    write, w_scale, _ = per_kernel(write_csv, "WRITE_SIZE")
    rec = {
        "source_digest": source_digest(),
        "workload": "wx256",
        "calibration": {"kernel": COPY_KERNEL, "bytes": COPY_BYTES,
                        "fetch_scale": round(f_scale, 4), "write_scale": round(w_scale, 4)},
        "kernels": {},
    }
    for k in sorted(set(fetch) & set(write)):
        rd, wr = fetch[k] * f_scale, write[k] * w_scale
        rec["kernels"][k] = {"fetch_kib": round(fetch[k] / 1024, 1),
                             "write_kib": round(write[k] / 1024, 1),
                             "hbm_read_bytes": int(rd), "hbm_write_bytes": int(wr),
                             "hbm_bytes_per_launch": int(rd + wr)}
    with open(out_path, "w") as f:
        json.dump(rec, f, indent=1)
        f.write("\n")
    return rec


def cpu_baseline(w, runs: int = 3):
    """The float64 oracle on the host cores, one whole layer call on the full
    workload (random complex input and filters of the workload's shapes: its
    cost does not depend on the values), `runs` times; median seconds."""
    import numpy as np
    import torch

    import oracle as O

    cores = len(os.sched_getaffinity(0))
    g = torch.Generator().manual_seed(7)

    def cn(*shape):
        z = torch.randn(*shape, 2, dtype=torch.float64, generator=g).numpy()
        return (z[..., 0] + 1j * z[..., 1]) / math.sqrt(2.0)

    x = cn(w.B, len(w.spins_in), w.C_in, w.H, w.W)
    K = cn(w.L, len(w.spins_out), w.C_out, len(w.spins_in), w.C_in)
    times = []
    for _ in range(runs):
        t0 = time.perf_counter()
        O.conv(x, K, w.L, w.spins_in, w.spins_out)
        times.append(time.perf_counter() - t0)
    t_layer = float(np.median(times))
    return {
        "value": 1.0 / t_layer,
        "unit": "fwd/s",
        "cores": cores,
        "kind": "oracle",
        "sample": (f"float64 numpy oracle (forward, mixing, inverse) on the full workload, "
                   f"{runs} layer calls, median {t_layer:.2f} s "
                   f"(runs: {', '.join(f'{t:.2f}' for t in times)} s)"),
        "seconds_per_fwd": t_layer,
        "cpu": _cpu_model(),
    }


def _cpu_model() -> str:
    try:
        for ln in open("/proc/cpuinfo"):
            if ln.startswith("model name"):
                return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="wx256")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a plain 1 GiB device copy (for counter calibration)")
    ap.add_argument("--summarize-counters", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="write profiles/traffic_<workload>.json from two counter runs and exit")
    args = ap.parse_args(argv)
    if args.summarize_counters:
        out = os.path.join(ROOT, "profiles", f"traffic_{args.workload}.json")
        print(json.dumps(summarize_counters(*args.summarize_counters, out)))
        return 0
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: the layer runs on one GPU only (it has no multi-GPU path); "
              "run with --gpus 1", file=sys.stderr)
        return 2

    import torch

    from paper_2306_05420_amd import swsft as S
    from paper_2306_05420_amd import synthetic as syn

    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        return 1
    w = syn.workload(args.workload)
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    plan = S.Plan(w.H, w.W, w.L, w.spins_in, w.spins_out, w.dtype)

    # inputs: band-limited fields synthesised on the GPU from seeded
    # CN(0,1)/(l+1) coefficients by the library's own inverse transform
    gen = torch.Generator(device=dev)
    gen.manual_seed(w.seed)
    decay = {"white": 0.0, "decay1": 1.0}.get(w.field, 1.0)
    coef = syn.torch_random_coefficients(gen, w.L, w.B, w.spins_in, w.C_in, decay)
    K = syn.torch_random_filters(gen, w.L, w.spins_in, w.C_in, w.spins_out, w.C_out,
                                 w.filter_var)
    if w.dtype == "bf16":
        coef = torch.view_as_real(coef).to(torch.bfloat16).contiguous()
        K = torch.view_as_real(K).to(torch.bfloat16).contiguous()
    plan_syn = S.Plan(w.H, w.W, w.L, w.spins_in, w.spins_in, w.dtype)
    x = plan_syn.inverse(coef)
    y = plan.empty(w.B, len(w.spins_out), w.C_out, w.H, w.W)
    torch.cuda.synchronize()
    plan_syn.close()
    del coef

    if args.copy_calibration:
        src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    for _ in range(args.warmup):
        plan.conv(x, K, y)
    torch.cuda.synchronize()

    # timed region: K layer calls
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    start.record()
    for _ in range(args.steps):
        plan.conv(x, K, y)
    stop.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    gpu_ms = start.elapsed_time(stop)
    elapsed = max(wall, gpu_ms / 1e3)
    ms_per_step = 1e3 * elapsed / args.steps
    value = args.steps / elapsed

    # per-stage HIP events over a second pass of K layer calls
    plan.stage_timing(True)
    for _ in range(args.steps):
        plan.conv(x, K, y)
    torch.cuda.synchronize()
    times = plan.stage_times()
    plan.stage_timing(False)

    work = stage_work(w)
    useful = sum(v["flops"] for v in work.values())
    stages = {}
    for name, (ms, n) in times.items():
        avg_s = ms / 1e3 / n
        rec = {"avg_us": round(avg_s * 1e6, 2), "launches": n}
        wk = work.get(name)
        if wk:
            rec["GB/s"] = round(wk["bytes"] / avg_s / 1e9, 1)
            rec["hbm_frac"] = round(wk["bytes"] / avg_s / 1e9 / HBM_PEAK_GBS, 4)
            if wk["flops"]:
                rec["TFLOP/s"] = round(wk["flops"] / avg_s / 1e12, 2)
                rec["mfma_frac"] = round(wk["flops"] / avg_s / 1e12 / PEAK_TFLOPS[w.dtype], 4)
        stages[name] = rec
    dom = max((k for k in stages if k in work), key=lambda k: stages[k]["avg_us"])
    avg_s = stages[dom]["avg_us"] / 1e6
    wk = work[dom]
    flops_per_byte = wk["flops"] / wk["bytes"]
    ridge = PEAK_TFLOPS[w.dtype] * 1e12 / (HBM_PEAK_GBS * 1e9)
    if wk["flops"] and flops_per_byte > ridge:
        roof = {"bound": "mfma", "achieved": round(wk["flops"] / avg_s / 1e12, 2),
                "peak": PEAK_TFLOPS[w.dtype], "unit": "TFLOP/s"}
    else:
        roof = {"bound": "hbm", "achieved": round(wk["bytes"] / avg_s / 1e9, 1),
                "peak": HBM_PEAK_GBS, "unit": "GB/s"}
    roof["frac"] = round(roof["achieved"] / roof["peak"], 4)
    roof["traffic"] = measured_traffic(dom)
    roof["kernel"] = dom
    roof["algorithmic_bytes_per_launch"] = wk["bytes"]
    roof["algorithmic_flops_per_launch"] = wk["flops"]

    tflops = useful / (elapsed / args.steps) / 1e12
    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "fwd/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {
            "workload": (f"{w.name}: {w.H}x{w.W} grid, L={w.L}, B={w.B}, spins "
                         f"{list(w.spins_in)}->{list(w.spins_out)}, C_in={w.C_in}, "
                         f"C_out={w.C_out}, {w.dtype} storage, fp32 accumulation"),
            "global_batch": w.B,
            "grid": [w.H, w.W],
            "bandlimit": w.L,
            "parallelism": "single GPU",
        },
        "tflops": round(tflops, 2),
        "mfma_peak_frac": round(tflops / PEAK_TFLOPS[w.dtype], 4),
        "useful_gflop_per_fwd": round(useful / 1e9, 3),
        "stages": stages,
        "roofline": roof,
    }
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w)
    plan.close()
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
