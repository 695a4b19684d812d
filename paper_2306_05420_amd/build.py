"""Build the HIP library libswsft.so in-tree for gfx950.

    python -m paper_2306_05420_amd.build        (or build() from Python)

Every HIP source is compiled with packed-FP32 instruction selection turned
off (packed FP32 instructions are avoided on this target) and -O3; objects go
to paper_2306_05420_amd/_build/.
"""

from __future__ import annotations

import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libswsft.so")
INCLUDE = os.path.join(os.path.dirname(PKG), "include")

SOURCES = ["tables.hip", "delta.hip", "dft.hip", "dft_mm.hip", "gemm.hip", "mix_dma.hip", "lat_dma.hip",
           "phase_collapse.hip", "batch_norm.hip", "backward.hip", "small.hip", "noalloc.hip",
           "probe.hip", "fused32.hip", "swsft_api.cpp"]
ARCH = "gfx950"


def _hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libswsft.so)")


def _compile(src: str, hipcc: str, build_dir: str = BUILD, defines=()) -> str:
    obj = os.path.join(build_dir, os.path.splitext(src)[0] + ".o")
    cmd = [hipcc, f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-Wall",
           "-Wno-unused-parameter", "-Wno-unused-variable",
           "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
           f"-I{INCLUDE}"] + [f"-D{d}" for d in defines] + ["-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"compile failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    noise = "not a recognized feature for this target"
    msgs = [ln for ln in (r.stderr or "").splitlines() if ln.strip() and noise not in ln]
    if msgs:
        sys.stderr.write("\n".join(msgs) + "\n")
    return obj


def build(verbose: bool = True, out: str = LIB, build_dir: str = BUILD, defines=()) -> str:
    """Compile every source and link libswsft.so; returns its path.  `defines`
    (NAME=VALUE strings) select tuning parameters for variant builds written
    to `out`."""
    hipcc = _hipcc()
    os.makedirs(build_dir, exist_ok=True)
    with ThreadPoolExecutor(max_workers=min(len(SOURCES), os.cpu_count() or 1)) as ex:
        objs = list(ex.map(lambda s: _compile(s, hipcc, build_dir, defines), SOURCES))
    tmp = out + ".tmp"
    cmd = [hipcc, f"--offload-arch={ARCH}", "-shared", "-fPIC", "-o", tmp] + objs
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed: {' '.join(cmd)}\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, out)
    if verbose:
        print(f"built {out}")
    return out


if __name__ == "__main__":
    build()
