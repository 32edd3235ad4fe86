"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer, on the CPU.

Two drivers in tests/sanitize/ run on exactly sized heap buffers so that any
out-of-bounds access, use after free, leak or undefined integer operation aborts
the run:
  oracle_asan.c  the CPU oracle (single messages of every length class with and
                 without AAD, both GF(2^128) multiplies; multi-chain round trips
                 with ragged last chains, 1 and 4 threads; tampered chains);
  host_asan.cpp  the library's host-only paths (the pipeline planner with exact
                 and short output arrays, the stage-size helper, the per-sample
                 chain layout, the chain count, the argument checks that return
                 before any HIP call). The library's sources are built with the
                 sanitizers on the host pass only; no device is touched.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = os.path.join(ROOT, "tests", "sanitize")
CSRC = os.path.join(ROOT, "paper_2410_15240_amd", "csrc")
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:halt_on_error=1",
           UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")


def run(cmd, **kw):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, **kw)
    return r.returncode, r.stdout


def test_oracle_under_asan_ubsan(tmp_path):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not found")
    exe = str(tmp_path / "oracle_asan")
    rc, out = run(["gcc", "-O1", "-g", "-std=c11", "-fopenmp", "-fno-omit-frame-pointer",
                   "-fsanitize=address,undefined", "-fno-sanitize-recover=all",
                   os.path.join(SAN, "oracle_asan.c"), os.path.join(ROOT, "oracle", "gcm_oracle.c"), "-o", exe])
    assert rc == 0, out
    rc, out = run([exe], env=dict(ENV, OMP_NUM_THREADS="4"), timeout=300)
    assert rc == 0 and "0 failures" in out and "Sanitizer" not in out, out[-4000:]


def test_library_host_paths_under_asan_ubsan(tmp_path):
    hipcc = "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not found")
    exe = str(tmp_path / "host_asan")
    rc, out = run([hipcc, "--offload-arch=gfx950", "-O1", "-g", "-std=c++17",
                   "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
                   "-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
                   "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer",
                   "-I", os.path.join(ROOT, "include"), "-I", CSRC,
                   os.path.join(SAN, "host_asan.cpp"), os.path.join(CSRC, "api.hip"),
                   os.path.join(CSRC, "kernels.hip"), os.path.join(CSRC, "bitslice.hip"), "-o", exe], timeout=600)
    assert rc == 0, out[-4000:]
    rc, out = run([exe], env=ENV, timeout=300)
    assert rc == 0 and "0 failures" in out and "Sanitizer" not in out, out[-4000:]
