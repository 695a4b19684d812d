"""The C-ABI layer (csrc/swsft_api.cpp) built for the host with
AddressSanitizer and UndefinedBehaviorSanitizer, against host stand-ins of
the HIP runtime and of the kernel launchers (tests/abi_host/hip_stub.cpp):
every entry point is called on buffers of exactly the documented sizes, each
launcher checks and touches the exact extent it would read or write, and
invalid calls must be refused.  Runs on the CPU; needs g++."""

import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)


@pytest.mark.skipif(shutil.which("g++") is None or not os.path.isdir("/opt/rocm/include"),
                    reason="needs g++ and the ROCm headers")
def test_abi_layer_under_address_and_ub_sanitizers(tmp_path):
    exe = str(tmp_path / "abi_host")
    cmd = ["g++", "-std=c++17", "-g", "-O1", "-fno-omit-frame-pointer",
           "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
           "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include", f"-I{ROOT}/include",
           os.path.join(ROOT, "paper_2306_05420_amd", "csrc", "swsft_api.cpp"),
           os.path.join(HERE, "abi_host", "hip_stub.cpp"),
           os.path.join(HERE, "abi_host", "abi_host_main.cpp"),
           "-o", exe, "-lpthread"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-4000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe], capture_output=True, text=True, env=env, timeout=600)
    print(r.stdout[-2000:])
    assert r.returncode == 0, (r.stdout[-2000:], r.stderr[-4000:])
    assert "ALL OK" in r.stdout
