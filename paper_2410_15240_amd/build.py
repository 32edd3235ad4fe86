"""Build the gfx950 HIP library in-tree: paper_2410_15240_amd/_lib/libfastrack.so.

    python -m paper_2410_15240_amd.build
"""
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
OUT_DIR = os.path.join(HERE, "_lib")
LIB = os.path.join(OUT_DIR, "libfastrack.so")
# Each source with the LLVM scheduling flags it is built with (see below).
SOURCES = [("kernels.hip", True), ("api.hip", True), ("bitslice.hip", False)]
ARCH = "gfx950"


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", "hipcc"):
        if cand and (os.path.sep not in cand or os.path.exists(cand)):
            return cand
    return "hipcc"


def build(verbose: bool = False) -> str:
    os.makedirs(OUT_DIR, exist_ok=True)
    tmp = LIB + ".tmp%d" % os.getpid()
    base = [hipcc(), "--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC", "-fvisibility=hidden",
            # keep hipcc from forming packed-FP32 instructions (this code has no FP, the flag is policy)
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-I", os.path.join(ROOT, "include"), "-I", CSRC]
    # LLVM's iterative max-occupancy scheduler keeps 4-8 table lookups in flight
    # per wave in the T-table AES rounds; the default strategy serialises them to
    # 1-2 once the kernel's live state grows. The bitsliced kernel (no lookups, a
    # 128-word state) is built with the default strategy, which keeps its rounds
    # free of register spills.
    maxocc = ["-mllvm", "--amdgpu-sched-strategy=iterative-maxocc"]
    noise = "is not a recognized feature for this target"
    objs, procs = [], []
    for src, sched in SOURCES:
        obj = os.path.join(OUT_DIR, src.replace(".hip", ".o.tmp%d" % os.getpid()))
        cmd = base + (maxocc if sched else []) + ["-c", os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((src, subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)))
        objs.append(obj)
    failed = []
    for src, pr in procs:
        out = "\n".join(l for l in pr.communicate()[0].splitlines() if noise not in l)
        if pr.returncode != 0:
            failed.append("hipcc failed on %s:\n%s" % (src, out))
        elif verbose and out.strip():
            print(out)
    if failed:   # no partial objects left behind in the package
        for o in objs:
            if os.path.exists(o):
                os.remove(o)
        raise RuntimeError("\n".join(failed))
    cmd = [hipcc(), "--offload-arch=" + ARCH, "-shared", "-fPIC"] + objs + ["-o", tmp, "-Wl,-rpath,/opt/rocm/lib"]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    for o in objs:
        os.remove(o)
    if r.returncode != 0:
        raise RuntimeError("hipcc link failed:\n" + r.stdout)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
    sys.exit(0)
