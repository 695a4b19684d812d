#!/usr/bin/env python3
"""Throughput of the spectral spin-weighted spherical convolution layer on one
MI355X: spin_sph_conv_forward on a 256 x 256 grid, bandlimit 128, batch 2,
spins {0,1} -> {0,1}, 256 -> 256 channels, bfloat16 storage with float32
accumulation (the large weather-shaped workload).

    python bench.py [--steps K] [--warmup W] [--gpus 1] [--no-cpu-baseline]
    python bench.py --table            (every workload: layer, transforms, backward, stack)
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
    # the synthesis runs over batch ranges whose spectrum fits 128 MiB of the
    # Infinity Cache (one range when the whole batch fits); each range's
    # launch reads the whole table
    per_item = So * M * Co * H * 2 * e
    bc = max(1, min(B, (128 << 20) // per_item)) if (So * 2 * Co * e) % 16 == 0 else B
    ranges = -(-B // bc)
    return {
        # small grids: whole transforms per map (the synthesis also mixes when
        # the layer runs without a separate mixing stage)
        "small_fwd": {"flops": lat_f, "bytes": x_b + tab_i + a_b},
        "small_inv": {"flops": lat_i, "bytes": a2_b + tab_o + y_b},
        "small_inv_mix": {"flops": lat_i + mix, "bytes": a_b + K_b + tab_o + y_b},
        "dft_fwd": {"flops": 0, "bytes": x_b + X_b},
        "lat_fwd": {"flops": lat_f, "bytes": X_b + tab_i + a_b},
        "mix": {"flops": mix, "bytes": a_b + K_b + a2_b},
        "lat_inv": {"flops": lat_i, "bytes": a2_b + ranges * tab_o + Y_b},
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


STAGE_KERNELS = re.compile(r"(dft_fwd|dft_inv|lat_fwd|lat_inv|mix)(?:_dma|_split)?_kernel")
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


def cpu_baseline(w, min_runs: int = 3, min_seconds: float = 10.0, max_runs: int = 200):
    """The float64 oracle on the host cores, whole layer calls on the full
    workload (random complex input and filters of the workload's shapes: its
    cost does not depend on the values), repeated until at least `min_runs`
    calls and `min_seconds` of work (a bounded sample); median seconds."""
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
    while len(times) < max_runs and (len(times) < min_runs or sum(times) < min_seconds):
        t0 = time.perf_counter()
        O.conv(x, K, w.L, w.spins_in, w.spins_out)
        times.append(time.perf_counter() - t0)
    runs = len(times)
    t_layer = float(np.median(times))
    return {
        "value": 1.0 / t_layer,
        "unit": "fwd/s",
        "cores": cores,
        "kind": "oracle",
        "sample": (f"float64 numpy oracle (forward, mixing, inverse) on the full workload, "
                   f"{runs} layer calls ({sum(times):.1f} s of work), median {t_layer:.3f} s "
                   f"(min {min(times):.3f}, max {max(times):.3f} s)"),
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


def vendor_mix(steps: int, warmup: int) -> dict:
    """The mixing stage at wx256 (L = 128, B = 2, spins {0,1}, C = 256) as real
    bf16 GEMMs per degree l, [2 (2l+1) B expanded rows x 2 S C] x [2 S C x S C],
    run by torch.bmm (hipBLASLt) with the rows padded to uniform batches: all
    degrees padded to 1024 rows, and degrees grouped by row counts padded to
    multiples of 256; next to spin_sph_mix on the same sizes (random values:
    timings do not depend on them)."""
    import torch

    from paper_2306_05420_amd import swsft as S

    dev = torch.device("cuda", 0)
    L, B, Sn, C = 128, 2, 2, 256
    Kp, N = 2 * Sn * C, Sn * C
    useful = sum(8 * (2 * l + 1) * B * N * N for l in range(L))

    def timed(fn):
        for _ in range(warmup):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(steps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / steps * 1e3  # us

    out = {"useful_gflop": round(useful / 1e9, 2)}
    a = torch.randn(L, 1024, Kp, device=dev).to(torch.bfloat16)
    b = torch.randn(L, Kp, N, device=dev).to(torch.bfloat16)
    us = timed(lambda: torch.bmm(a, b))
    out["bmm_padded_1024"] = {"us": round(us, 1), "useful_TFLOP/s": round(useful / us / 1e6, 1)}
    del a, b
    groups = {}
    for l in range(L):
        groups.setdefault((2 * (2 * l + 1) * B + 255) // 256 * 256, []).append(l)
    mats = [(torch.randn(len(ls), g, Kp, device=dev).to(torch.bfloat16),
             torch.randn(len(ls), Kp, N, device=dev).to(torch.bfloat16)) for g, ls in groups.items()]
    us = timed(lambda: [torch.bmm(x, y) for x, y in mats])
    out["bmm_grouped_256"] = {"us": round(us, 1), "useful_TFLOP/s": round(useful / us / 1e6, 1),
                              "launches": len(mats)}
    del mats
    plan = S.Plan(2 * L, 2 * L, L, (0, 1), (0, 1), "bf16")
    coef = plan.empty(L * L, B, Sn, C)
    coef.copy_(torch.randn(coef.shape, device=dev).to(torch.bfloat16))
    K = plan.empty(L, Sn, C, Sn, C)
    K.copy_(torch.randn(K.shape, device=dev).to(torch.bfloat16))
    res = plan.empty(L * L, B, Sn, C)
    us = timed(lambda: plan.mix(coef, K, res))
    out["spin_sph_mix"] = {"us": round(us, 1), "useful_TFLOP/s": round(useful / us / 1e6, 1)}
    plan.close()
    return out


def main(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default="wx256")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--forward-only", action="store_true",
                    help="time the layer and the transforms only (no backward or graph replay "
                         "timing): the launches that profiling runs attribute to the layer")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run a plain 1 GiB device copy (for counter calibration)")
    ap.add_argument("--table", action="store_true",
                    help="measure every workload and print markdown table rows")
    ap.add_argument("--dft-vs-fft", action="store_true",
                    help="compare the FFT and the DFT-matrix forward longitude stages at "
                         "256^2, 512^2 and 768^2 (B = 1, spins {0,1}, C = 256, bf16)")
    ap.add_argument("--delta-routes", action="store_true",
                    help="compare the latitude stages: direct d(theta) tables vs the Wigner-Delta "
                         "route with and without its symmetries (wx128 and wx256 workloads)")
    ap.add_argument("--vendor-mix", action="store_true",
                    help="time torch's bf16 batched matmul (hipBLASLt) on the mixing stage's "
                         "per-degree shapes at wx256 next to the library's mixing kernel")
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

    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        return 1
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    if args.delta_routes:
        print(DELTA_HEAD)
        for name in ("wx128", "wx256"):
            for route in ("direct", "delta_sym", "delta"):
                print(delta_route_row(name, route, min(args.steps, 50), min(args.warmup, 5)),
                      flush=True)
        return 0
    if args.vendor_mix:
        print(json.dumps(vendor_mix(min(args.steps, 50), min(args.warmup, 5))))
        return 0
    if args.dft_vs_fft:
        print(DFT_HEAD)
        for H in (256, 512, 768):
            for method in ("fft", "matmul"):
                print(dft_vs_fft_row(H, method, min(args.steps, 50), min(args.warmup, 5)),
                      flush=True)
        print()
        print(DFT_LAYER_HEAD)
        for H in (256, 512, 768):
            for method in ("fft", "matmul"):
                print(dft_vs_fft_layer_row(H, method, min(args.steps, 20), min(args.warmup, 3)),
                      flush=True)
        return 0
    if args.table:
        from paper_2306_05420_amd import synthetic as syn
        print(TABLE_HEAD)
        for i, wl in enumerate(syn.WORKLOADS):
            # launch-bound workloads (a few µs per call) get 1000 timed calls
            steps = 1000 if wl.name in ("tiny", "small") else min(args.steps, 100)
            r = measure(wl.name, steps, min(args.warmup, 10), dev)
            for row in table_rows(i + 1, r):
                print(row, flush=True)
        return 0

    r = measure(args.workload, args.steps, args.warmup, dev, args.copy_calibration,
                extras=not args.forward_only)
    w = r["w"]
    out = {
        "metric": METRIC,
        "value": round(r["value"], 2),
        "unit": "fwd/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(r["ms_per_step"], 4),
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
        "latency_us": r["latency_us"],
        "tflops": round(r["tflops"], 2),
        "mfma_peak_frac": round(r["tflops"] / PEAK_TFLOPS[w.dtype], 4),
        "useful_gflop_per_fwd": round(r["useful"] / 1e9, 3),
        "stages": r["stages"],
        "roofline": r["roofline"],
        "transforms": r["transforms"],
        "plan_ms": r["plan_ms"],
    }
    for k in ("backward", "graph"):
        if k in r:
            out[k] = r[k]
    if not args.forward_only:
        out["measured_peaks"] = measured_peaks()
    if "stack2" in r:
        out["stack2"] = r["stack2"]
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(w)
    print(json.dumps(out), flush=True)
    return 0


def measured_peaks() -> dict:
    """Achievable peaks on this GPU in the same run, for context next to the
    datasheet figures: a plain 1 GiB device-to-device copy (bytes read +
    written per second) and a large bf16 GEMM through the vendor library."""
    import torch

    src = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    t_copy = _time_calls(lambda: dst.copy_(src), 10, 3)
    del src, dst
    n = 8192
    a = torch.randn((n, n), device="cuda").to(torch.bfloat16)
    b = torch.randn((n, n), device="cuda").to(torch.bfloat16)
    c = torch.empty((n, n), device="cuda", dtype=torch.bfloat16)
    t_mm = _time_calls(lambda: torch.matmul(a, b, out=c), 10, 3)
    del a, b, c
    out = {"copy_GB/s": round(2 * (1 << 30) / t_copy / 1e9, 1),
           "bf16_gemm_TFLOP/s": round(2.0 * n ** 3 / t_mm / 1e12, 1),
           "gemm": f"torch.matmul bf16 {n}x{n}x{n}"}
    out.update(mfma_probe_rates())
    return out


def mfma_probe_rates() -> dict:
    """The library's register-only MFMA probe (swsft_probe_mfma): 2,048 waves
    (two per SIMD) of four independent MFMA chains, timed with events on the
    stream it runs on; TFLOP/s for bf16 32x32x16 with random and with
    constant operands, and for f32 32x32x2 with random operands."""
    import torch

    from paper_2306_05420_amd import swsft as S

    n_waves = 2048
    buf = torch.empty(64 * n_waves, dtype=torch.float32, device="cuda")
    rates = {}
    for key, dtype, rnd, iters in (("bf16_mfma_random_TFLOP/s", "bf16", True, 20000),
                                   ("bf16_mfma_constant_TFLOP/s", "bf16", False, 20000),
                                   ("f32_mfma_random_TFLOP/s", "f32", True, 10000)):
        flops = S.probe_mfma(dtype, rnd, iters, n_waves, buf)  # warm-up
        t = _time_calls(lambda: S.probe_mfma(dtype, rnd, iters, n_waves, buf), 5, 1)
        if not bool(torch.isfinite(buf).all()):
            raise RuntimeError("MFMA probe produced non-finite checksums")
        rates[key] = round(flops / t / 1e12, 1)
    rates["mfma_probe"] = f"{n_waves} waves x 4 register-only MFMA chains (swsft_probe_mfma)"
    return rates


def _time_calls(fn, steps: int, warmup: int):
    """Seconds per call of fn over `steps` calls after `warmup`, bracketed by
    device synchronizations: the larger of wall clock and stream events."""
    import torch

    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    start = torch.cuda.Event(enable_timing=True)
    stop = torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    start.record()
    for _ in range(steps):
        fn()
    stop.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    return max(wall, start.elapsed_time(stop) / 1e3) / steps


def _time_graph(fn, steps: int, warmup: int):
    """Seconds per replay of a HIP graph holding one call of fn."""
    import torch

    fn()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fn()
    torch.cuda.current_stream().wait_stream(side)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    t = _time_calls(g.replay, steps, warmup)
    del g
    return t


def measure(name: str, steps: int, warmup: int, dev, copy_calibration: bool = False,
            extras: bool = True) -> dict:
    """Time one workload: the layer (with per-stage HIP events and the
    roofline of its dominant stage), the forward and inverse transforms alone,
    and for the molecule workload the two-layer stack with phase collapse."""
    import torch

    from paper_2306_05420_amd import swsft as S
    from paper_2306_05420_amd import synthetic as syn

    w = syn.workload(name)
    # plan creation (device tables and twiddles), outside every timed loop
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    plan = S.Plan(w.H, w.W, w.L, w.spins_in, w.spins_out, w.dtype)
    torch.cuda.synchronize()
    plan_ms = (time.perf_counter() - t0) * 1e3

    # inputs: band-limited fields synthesised on the GPU from seeded
    # CN(0,1)/(l+1) coefficients by the library's own inverse transform
    gen = torch.Generator(device=dev)
    gen.manual_seed(w.seed)
    decay = {"white": 0.0, "decay1": 1.0}.get(w.field, 1.0)

    def storage(t):
        return torch.view_as_real(t).to(torch.bfloat16).contiguous() if w.dtype == "bf16" else t

    coef = storage(syn.torch_random_coefficients(gen, w.L, w.B, w.spins_in, w.C_in, decay))
    K = storage(syn.torch_random_filters(gen, w.L, w.spins_in, w.C_in, w.spins_out, w.C_out,
                                         w.filter_var))
    coef_out = storage(syn.torch_random_coefficients(gen, w.L, w.B, w.spins_out, w.C_out, decay))
    plan_syn = S.Plan(w.H, w.W, w.L, w.spins_in, w.spins_in, w.dtype)
    x = plan_syn.inverse(coef)
    y = plan.empty(w.B, len(w.spins_out), w.C_out, w.H, w.W)
    torch.cuda.synchronize()
    plan_syn.close()

    if copy_calibration:
        src = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    # timed region: K layer calls
    t_layer = _time_calls(lambda: plan.conv(x, K, y), steps, warmup)
    # per-call latency distribution (a separate pass, one event pair per call)
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(steps)]
    for e0, e1 in evs:
        e0.record()
        plan.conv(x, K, y)
        e1.record()
    torch.cuda.synchronize()
    per_call = sorted(e0.elapsed_time(e1) * 1e3 for e0, e1 in evs)
    pct = lambda q: round(per_call[min(len(per_call) - 1, int(q * len(per_call)))], 2)
    latency = {"p10": pct(0.1), "p50": pct(0.5), "p90": pct(0.9)}

    # per-stage HIP events over a second pass of K layer calls
    plan.stage_timing(True)
    for _ in range(steps):
        plan.conv(x, K, y)
    torch.cuda.synchronize()
    times = plan.stage_times()
    plan.stage_timing(False)

    work = stage_work(w)
    useful = sum(work[k]["flops"] for k in ("lat_fwd", "mix", "lat_inv"))
    if "mix" not in times:  # small grids: the synthesis kernel mixes as well
        work["small_inv"] = work["small_inv_mix"]
    stages = {}
    for sname, (ms, n) in times.items():
        # a stage may run as several launches per call (the inverse stages over
        # batch ranges): avg_us is per launch, us_per_call per layer call
        call_s = ms / 1e3 / steps
        rec = {"avg_us": round(ms * 1e3 / n, 2), "launches_per_call": round(n / steps, 3),
               "us_per_call": round(call_s * 1e6, 2)}
        wk = work.get(sname)
        if wk:
            rec["GB/s"] = round(wk["bytes"] / call_s / 1e9, 1)
            rec["hbm_frac"] = round(wk["bytes"] / call_s / 1e9 / HBM_PEAK_GBS, 4)
            if wk["flops"]:
                rec["TFLOP/s"] = round(wk["flops"] / call_s / 1e12, 2)
                rec["mfma_frac"] = round(wk["flops"] / call_s / 1e12 / PEAK_TFLOPS[w.dtype], 4)
        stages[sname] = rec
    dom = max((k for k in stages if k in work), key=lambda k: stages[k]["us_per_call"])
    lpc = times[dom][1] / steps
    avg_s = stages[dom]["avg_us"] / 1e6          # one launch
    wk = {k: v / lpc for k, v in work[dom].items()}  # one launch's share of the stage
    flops_per_byte = wk["flops"] / wk["bytes"]
    ridge = PEAK_TFLOPS[w.dtype] * 1e12 / (HBM_PEAK_GBS * 1e9)
    if wk["flops"] and flops_per_byte > ridge:
        roof = {"bound": "mfma", "achieved": round(wk["flops"] / avg_s / 1e12, 2),
                "peak": PEAK_TFLOPS[w.dtype], "unit": "TFLOP/s"}
    else:
        roof = {"bound": "hbm", "achieved": round(wk["bytes"] / avg_s / 1e9, 1),
                "peak": HBM_PEAK_GBS, "unit": "GB/s"}
    roof["frac"] = round(roof["achieved"] / roof["peak"], 4)
    roof["traffic"] = measured_traffic(dom) if name == "wx256" else None
    roof["kernel"] = dom
    roof["algorithmic_bytes_per_launch"] = int(wk["bytes"])
    roof["algorithmic_flops_per_launch"] = int(wk["flops"])
    roof["launches_per_call"] = round(lpc, 3)

    # the transforms alone: forward on x (input spins), inverse on a
    # coefficient set of the output spins
    coef_f = plan.forward(x)
    y_i = plan.empty(w.B, len(w.spins_out), w.C_out, w.H, w.W)
    t_fwd = _time_calls(lambda: plan.forward(x, coef_f), steps, warmup)
    t_inv = _time_calls(lambda: plan.inverse(coef_out, y_i), steps, warmup)
    transforms = {}
    work = stage_work(w)
    small = "small_fwd" in times
    for tname, t, keys in (("forward", t_fwd, ("small_fwd",) if small else ("dft_fwd", "lat_fwd")),
                           ("inverse", t_inv, ("small_inv",) if small else ("lat_inv", "dft_inv"))):
        byt = sum(work[k]["bytes"] for k in keys)
        fl = sum(work[k]["flops"] for k in keys)
        transforms[tname] = {"us": round(t * 1e6, 2), "per_s": round(1.0 / t, 1),
                             "GB/s": round(byt / t / 1e9, 1),
                             "TFLOP/s": round(fl / t / 1e12, 2)}
    r = {"w": w, "value": 1.0 / t_layer, "ms_per_step": t_layer * 1e3, "latency_us": latency,
         "tflops": useful / t_layer / 1e12, "useful": useful, "stages": stages,
         "roofline": roof, "transforms": transforms, "plan_ms": round(plan_ms, 2)}
    if not extras:
        plan.close()
        return r
    r["backward"] = measure_backward(plan, w, x, K, y, steps, warmup)
    # launch overhead removed: one layer call (and one backward call) per
    # replay of a captured graph
    gx = plan.empty(w.B, len(w.spins_in), w.C_in, w.H, w.W)
    gk = plan.empty(w.L, len(w.spins_out), w.C_out, len(w.spins_in), w.C_in)
    y_g = plan.empty(w.B, len(w.spins_out), w.C_out, w.H, w.W)
    t_gl = _time_graph(lambda: plan.conv(x, K, y_g), steps, warmup)
    t_gb = _time_graph(lambda: plan.conv_backward(x, K, y, grad_x=gx, grad_filters=gk),
                       steps, warmup)
    r["graph"] = {"layer_us": round(t_gl * 1e6, 2), "layer_per_s": round(1.0 / t_gl, 1),
                  "backward_us": round(t_gb * 1e6, 2)}
    del gx, gk, y_g

    if name == "mol":
        # two stacked layers with the phase collapse between them
        plan2 = S.Plan(w.H, w.W, w.L, w.spins_out, w.spins_out, w.dtype)
        K2 = storage(syn.torch_random_filters(gen, w.L, w.spins_out, w.C_out, w.spins_out,
                                              w.C_out, w.filter_var))
        So = len(w.spins_out)
        W1 = syn.torch_complex_normal(gen, (w.C_out, w.C_out), 1.0 / w.C_out)
        W2 = syn.torch_complex_normal(gen, (w.C_out, So * w.C_out), 1.0 / (So * w.C_out))
        bias = syn.torch_complex_normal(gen, (w.C_out,), 0.01)
        z = plan.empty(w.B, So, w.C_out, w.H, w.W)
        y2 = plan.empty(w.B, So, w.C_out, w.H, w.W)

        def stack():
            plan.conv(x, K, y)
            plan.phase_collapse(y, W1, W2, bias, y=z)
            plan2.conv(z, K2, y2)

        t2 = _time_calls(stack, steps, warmup)
        r["stack2"] = {"us": round(t2 * 1e6, 2), "per_s": round(1.0 / t2, 1),
                       "TFLOP/s": round(2 * useful / t2 / 1e12, 2)}
        plan2.close()
        r["block"] = {f"{hi}to{ho}": measure_block(w, hi, ho, gen, storage, steps, warmup)
                      for hi, ho in ((w.H, w.H), (2 * w.H, w.H))}
    plan.close()
    return r


DELTA_HEAD = ("| workload | latitude route | swsft_forward µs | swsft_inverse µs | layer µs | "
              "latitude-stage µs (fwd + inv, incl. theta GEMMs) | vs direct (layer) |\n"
              "|---|---|---|---|---|---|---|")
_DELTA_BASE = {}


def delta_route_row(name: str, route: str, steps: int, warmup: int) -> str:
    """Forward, inverse and layer times of a workload with the latitude stages
    by the direct d(theta) tables or by the Wigner-Delta route (eqs. (4)-(6))
    without ("delta") or with ("delta_sym") its J / G symmetries."""
    import torch

    from paper_2306_05420_amd import swsft as S
    from paper_2306_05420_amd import synthetic as syn

    w = syn.workload(name)
    plan = S.Plan(w.H, w.W, w.L, w.spins_in, w.spins_out, w.dtype, latitude=route)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(w.seed)

    def storage(t):
        return torch.view_as_real(t).to(torch.bfloat16).contiguous() if w.dtype == "bf16" else t

    x = storage(syn.torch_complex_normal(gen, (w.B, len(w.spins_in), w.C_in, w.H, w.W)))
    K = storage(syn.torch_random_filters(gen, w.L, w.spins_in, w.C_in, w.spins_out, w.C_out,
                                         w.filter_var))
    a = storage(syn.torch_random_coefficients(gen, w.L, w.B, w.spins_out, w.C_out, 1.0))
    coef = plan.forward(x)
    y = plan.inverse(a)
    yc = plan.conv(x, K)
    t_f = _time_calls(lambda: plan.forward(x, coef), steps, warmup)
    t_i = _time_calls(lambda: plan.inverse(a, y), steps, warmup)
    t_c = _time_calls(lambda: plan.conv(x, K, yc), steps, warmup)
    plan.stage_timing(True)
    for _ in range(steps):
        plan.conv(x, K, yc)
    torch.cuda.synchronize()
    st = plan.stage_times()
    plan.stage_timing(False)
    plan.close()
    lat = sum(st[k][0] for k in ("lat_fwd", "lat_inv", "delta_theta") if k in st) * 1e3 / steps
    if route == "direct":
        _DELTA_BASE[name] = t_c
    rel = f"{t_c / _DELTA_BASE[name]:.2f}×" if name in _DELTA_BASE else "—"
    return (f"| {name} | {route} | {t_f * 1e6:.1f} | {t_i * 1e6:.1f} | {t_c * 1e6:.1f} | "
            f"{lat:.1f} | {rel} |")


DFT_HEAD = ("| grid | forward longitude stage | longitude µs | GB/s | DFT-matmul TFLOP/s | "
            "% bf16 peak | whole forward transform µs | same GEMM in torch.matmul µs |\n"
            "|---|---|---|---|---|---|---|---|")


def dft_vs_fft_row(H: int, method: str, steps: int, warmup: int) -> str:
    """Forward transform of one batch item (spins {0,1}, C = 256, bf16) on an
    H x H grid with bandlimit H/2, with the register-FFT or the DFT-matrix
    longitude stage: the longitude stage alone (HIP events) and the whole
    swsft_forward.  The FFT route takes powers of two up to 512 only."""
    import torch

    from paper_2306_05420_amd import swsft as S
    from paper_2306_05420_amd import synthetic as syn

    B, spins, C, L = 1, (0, 1), 256, H // 2
    pow2 = H & (H - 1) == 0 and H <= 512
    if method == "fft" and not pow2:
        return f"| {H}² | register FFT | — (no FFT of this width) | — | — | — | — | — |"
    plan = S.Plan(H, H, L, spins, spins, "bf16", longitude=method)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(H)
    x = torch.view_as_real(syn.torch_complex_normal(gen, (B, 2, C, H, H))).to(
        torch.bfloat16).contiguous()
    coef = plan.forward(x)
    t = _time_calls(lambda: plan.forward(x, coef), steps, warmup)
    plan.stage_timing(True)
    for _ in range(steps):
        plan.forward(x, coef)
    torch.cuda.synchronize()
    st = plan.stage_times()
    plan.stage_timing(False)
    plan.close()
    lon = st["dft_fwd"][0] / st["dft_fwd"][1] / 1e3  # seconds
    M = 2 * L - 1
    lib = "—"
    if method == "matmul":
        # the same real GEMM [rows x 2W] . [2W x 2M] through the vendor library
        # (row-major output, without the scatter into the K-tiled spectrum)
        Ft = torch.randn((2 * H, 2 * M), generator=gen, device="cuda").to(torch.bfloat16)
        xm = x.view(B * 2 * C * H, 2 * H)
        out = torch.empty((xm.shape[0], 2 * M), dtype=torch.bfloat16, device="cuda")
        lib = f"{_time_calls(lambda: torch.matmul(xm, Ft, out=out), steps, warmup) * 1e6:.1f}"
        del Ft, out
    rows = B * 2 * C * H
    byt = rows * H * 4 + 2 * M * B * C * H * 4        # x in, X out (bf16 pairs)
    fl = 2.0 * rows * (2 * H) * (2 * M)                # the dense real GEMM
    name = "register FFT (VALU)" if method == "fft" else "DFT matrix (MFMA bf16)"
    tf = f"{fl / lon / 1e12:.0f}" if method == "matmul" else "—"
    pk = f"{100 * fl / lon / 1e12 / PEAK_TFLOPS['bf16']:.1f}" if method == "matmul" else "—"
    return (f"| {H}² | {name} | {lon * 1e6:.1f} | {byt / lon / 1e9:.0f} | {tf} | {pk} | "
            f"{t * 1e6:.1f} | {lib} |")


DFT_LAYER_HEAD = ("| grid | longitude stages | layer µs | forward longitude µs | "
                  "inverse longitude µs (per call) | layer vs FFT route |\n"
                  "|---|---|---|---|---|---|")
_DFT_LAYER_BASE = {}


def dft_vs_fft_layer_row(H: int, method: str, steps: int, warmup: int) -> str:
    """The whole layer (B = 1, spins {0,1} -> {0,1}, C = 256 -> 256, bf16,
    bandlimit H/2) with the register-FFT or the DFT-matrix longitude stages in
    both directions: layer time and the two longitude stages (HIP events)."""
    import torch

    from paper_2306_05420_amd import swsft as S
    from paper_2306_05420_amd import synthetic as syn

    B, spins, C, L = 1, (0, 1), 256, H // 2
    pow2 = H & (H - 1) == 0 and H <= 512
    if method == "fft" and not pow2:
        return f"| {H}² | register FFT | — (no FFT of this width) | — | — | — |"
    plan = S.Plan(H, H, L, spins, spins, "bf16", longitude=method)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(H + 1)
    x = torch.view_as_real(syn.torch_complex_normal(gen, (B, 2, C, H, H))).to(
        torch.bfloat16).contiguous()
    K = torch.view_as_real(syn.torch_random_filters(gen, L, spins, C, spins, C, 1.0 / (2 * C))).to(
        torch.bfloat16).contiguous()
    y = plan.conv(x, K)
    t = _time_calls(lambda: plan.conv(x, K, y), steps, warmup)
    plan.stage_timing(True)
    for _ in range(steps):
        plan.conv(x, K, y)
    torch.cuda.synchronize()
    st = plan.stage_times()
    plan.stage_timing(False)
    plan.close()
    fwd = st["dft_fwd"][0] / steps * 1e3
    inv = st["dft_inv"][0] / steps * 1e3
    if method == "fft":
        _DFT_LAYER_BASE[H] = t
    rel = f"{t / _DFT_LAYER_BASE[H]:.2f}×" if H in _DFT_LAYER_BASE else "—"
    name = "register FFT (VALU)" if method == "fft" else "DFT matrices (MFMA bf16)"
    return f"| {H}² | {name} | {t * 1e6:.1f} | {fwd:.1f} | {inv:.1f} | {rel} |"


def block_flops(w, H_in: int, H_out: int) -> int:
    """Useful flops of one residual-block call on spins_out x C_out channels:
    one forward-latitude contraction on the input grid, one on the output
    grid, two inverse-latitude contractions and two mixings."""
    L, B, C = w.L, w.B, w.C_out
    lat = lambda H: sum(4 * H * B * C * (L * L - s * s) for s in w.spins_out)
    mix = 0
    for l in range(L):
        k = C * sum(1 for s in w.spins_out if abs(s) <= l)
        mix += 8 * B * (2 * l + 1) * k * k
    return lat(H_in) + 3 * lat(H_out) + 2 * mix


def measure_block(w, H_in: int, H_out: int, gen, storage, steps: int, warmup: int) -> dict:
    """Time the residual block (spins_out -> spins_out, C_out channels) from an
    H_in grid to an H_out grid (spectral pooling when H_out < H_in)."""
    import torch

    from paper_2306_05420_amd import swsft as S
    from paper_2306_05420_amd import synthetic as syn

    spins, C, B, L = w.spins_out, w.C_out, w.B, w.L
    Sn = len(spins)
    blk = S.ResidualBlock(H_in, H_out, spins, C, w.dtype, L=L)
    x = storage(syn.torch_complex_normal(gen, (B, Sn, C, H_in, H_in)))
    K1 = storage(syn.torch_random_filters(gen, L, spins, C, spins, C, w.filter_var))
    K2 = storage(syn.torch_random_filters(gen, L, spins, C, spins, C, w.filter_var))
    dev = x.device
    g1 = torch.ones((Sn, C), dtype=torch.float32, device=dev)
    g2 = torch.ones((Sn, C), dtype=torch.float32, device=dev)
    b1 = syn.torch_complex_normal(gen, (C,), 0.01)
    b2 = syn.torch_complex_normal(gen, (C,), 0.01)
    pc = lambda: (syn.torch_complex_normal(gen, (C, C), 1.0 / C),
                  syn.torch_complex_normal(gen, (C, Sn * C), 1.0 / (Sn * C)),
                  syn.torch_complex_normal(gen, (C,), 0.01))
    pc1, pc2 = pc(), pc()
    y = blk.p_out.empty(B, Sn, C, H_out, H_out)
    fn = lambda: blk.forward(x, K1, K2, g1, b1, g2, b2, pc1, pc2, 1e-5, y=y)
    t = _time_calls(fn, steps, warmup)
    blk.p_out.stage_timing(True)
    for _ in range(steps):
        fn()
    torch.cuda.synchronize()
    times = blk.p_out.stage_times()
    blk.p_out.stage_timing(False)
    blk.close()
    fl = block_flops(w, H_in, H_out)
    e = 2 if w.dtype == "bf16" else 4
    coef_b = L * L * B * Sn * C * 2 * e
    stages = {k: {"us_per_call": round(ms * 1e3 / steps, 2), "launches_per_call": n // steps}
              for k, (ms, n) in times.items()}
    if "batch_norm" in stages:
        # per call: two norms, each reading its input twice and writing once, the
        # second also reading the skip coefficients
        bn_bytes = 7 * coef_b
        stages["batch_norm"]["GB/s"] = round(bn_bytes / (stages["batch_norm"]["us_per_call"] * 1e3), 1)
    return {"grid": f"{H_in}x{H_in} -> {H_out}x{H_out}", "us": round(t * 1e6, 2),
            "per_s": round(1.0 / t, 1), "TFLOP/s": round(fl / t / 1e12, 2),
            "useful_gflop": round(fl / 1e9, 3), "stages": stages}


def backward_flops(w) -> int:
    """Useful flops of one backward call (both gradients): G^H on the output
    gradient and F on x (forward-transform contractions), the filter gradient
    and the adjoint mixing (each as many as the mixing), F^H (an inverse
    contraction over the input spins)."""
    work = stage_work(w)
    H, L, B = w.H, w.L, w.B
    lat_out = sum(4 * H * B * w.C_out * (L * L - t * t) for t in w.spins_out)
    return 2 * work["lat_fwd"]["flops"] + lat_out + 2 * work["mix"]["flops"]


def measure_backward(plan, w, x, K, grad_y, steps: int, warmup: int) -> dict:
    """Time spin_sph_conv_backward (grad_x and grad_filters) with per-stage
    HIP events over a second pass."""
    import torch

    gx = plan.empty(w.B, len(w.spins_in), w.C_in, w.H, w.W)
    gk = plan.empty(w.L, len(w.spins_out), w.C_out, len(w.spins_in), w.C_in)
    fn = lambda: plan.conv_backward(x, K, grad_y, grad_x=gx, grad_filters=gk)
    t = _time_calls(fn, steps, warmup)
    plan.stage_timing(True)
    for _ in range(steps):
        fn()
    torch.cuda.synchronize()
    times = plan.stage_times()
    plan.stage_timing(False)
    fl = backward_flops(w)
    # per call: stage -> (microseconds, launches)
    stages = {k: {"us_per_call": round(ms * 1e3 / steps, 2), "launches_per_call": n // steps}
              for k, (ms, n) in times.items()}
    # training: the forward saves the input's coefficients, the backward reuses them
    _, cx = plan.conv(x, K, coef_x=True)
    t_saved = _time_calls(lambda: plan.conv_backward(x, K, grad_y, grad_x=gx, grad_filters=gk,
                                                     coef_x=cx), steps, warmup)
    return {"us": round(t * 1e6, 2), "per_s": round(1.0 / t, 1),
            "TFLOP/s": round(fl / t / 1e12, 2), "useful_gflop": round(fl / 1e9, 3),
            "stages": stages, "us_with_saved_coefficients": round(t_saved * 1e6, 2)}


TABLE_HEAD = ("| Cfg | Op | median µs | calls/s | useful TFLOP/s | % MFMA peak | "
              "GB/s (DFT stages fwd / inv) | % HBM roofline (dominant stage) |\n"
              "|---|---|---|---|---|---|---|---|")


def table_rows(cfg: int, r: dict):
    w, st = r["w"], r["stages"]
    peak = PEAK_TFLOPS[w.dtype]
    if "dft_fwd" in st:
        dft = f"{st['dft_fwd']['GB/s']:.0f} / {st['dft_inv']['GB/s']:.0f}"
    else:
        dft = f"{st['small_fwd']['GB/s']:.0f} / {st['small_inv']['GB/s']:.0f} (whole transforms)"
    roof = f"{100 * r['roofline']['frac']:.1f} ({r['roofline']['kernel']})"
    rows = [f"| {cfg} {w.name} | layer | {r['ms_per_step'] * 1e3:.1f} | {r['value']:.0f} | "
            f"{r['tflops']:.1f} | {100 * r['tflops'] / peak:.1f} | {dft} | {roof} |"]
    for op in ("forward", "inverse"):
        t = r["transforms"][op]
        rows.append(f"| {cfg} {w.name} | swsft_{op} | {t['us']:.1f} | {t['per_s']:.0f} | "
                    f"{t['TFLOP/s']:.1f} | {100 * t['TFLOP/s'] / peak:.1f} | {t['GB/s']:.0f} (whole transform) | — |")
    t = r["graph"]
    rows.append(f"| {cfg} {w.name} | layer, HIP graph replay | {t['layer_us']:.1f} | "
                f"{t['layer_per_s']:.0f} | {r['useful'] / t['layer_us'] / 1e6:.1f} | "
                f"{100 * r['useful'] / t['layer_us'] / 1e6 / peak:.1f} | — | — |")
    t = r["backward"]
    rows.append(f"| {cfg} {w.name} | layer backward (grad_x, grad_filters) | {t['us']:.1f} | "
                f"{t['per_s']:.0f} | {t['TFLOP/s']:.1f} | {100 * t['TFLOP/s'] / peak:.1f} | — | — |")
    if "stack2" in r:
        t = r["stack2"]
        rows.append(f"| {cfg} {w.name} | 2 layers + phase collapse | {t['us']:.1f} | {t['per_s']:.0f} | "
                    f"{t['TFLOP/s']:.1f} | {100 * t['TFLOP/s'] / peak:.1f} | — | — |")
    for t in r.get("block", {}).values():
        rows.append(f"| {cfg} {w.name} | residual block {t['grid']} | {t['us']:.1f} | {t['per_s']:.0f} | "
                    f"{t['TFLOP/s']:.1f} | {100 * t['TFLOP/s'] / peak:.1f} | — | — |")
    return rows


if __name__ == "__main__":
    sys.exit(main())
