"""Build the native library libnv.so (HIP for gfx950) in-tree.

Usage: python paper_2312_04429_amd/build.py   (by path: importing the package
loads libnv.so, which may be stale or missing before the build)
"""
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.environ.get("NV_BUILD_SRC") or os.path.join(HERE, "csrc")
OUT_DIR = os.environ.get("NV_BUILD_DIR") or os.path.join(HERE, "_build")
LIB = os.environ.get("NV_BUILD_OUT") or os.path.join(HERE, "libnv.so")
SOURCES = ["lookup.hip", "gemm.hip", "attention.hip", "ops.hip", "unet.hip", "trace.hip",
           "probe.hip", "pool.hip", "lcbfu.cpp", "predictor.hip", "ivf.hip"]
ARCH = os.environ.get("NV_OFFLOAD_ARCH", "gfx950")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
         # packed fp32 ops stay off: the compiler would otherwise form v_pk_* fp32 math
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wno-pass-failed"]


# Per-source flags.  attention.hip: matrix instructions write VGPRs (its
# softmax reads every score back; the accumulator-register form adds a copy
# per score).  probe.hip: the same form, which is what reaches the matrix
# cores' rate in a pure multiply loop (about 2.2 PFLOP/s against 1.2 with
# accumulators in AGPRs).
# predictor.hip, ivf.hip: no multiply-add contraction, so their float64 sums
# round exactly as written.
EXTRA = {"attention.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"],
         "probe.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"],
         "predictor.hip": ["-ffp-contract=off"],
         "ivf.hip": ["-ffp-contract=off"]}


def _compile(src):
    obj = os.path.join(OUT_DIR, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, *FLAGS, *EXTRA.get(src, []), "-c", os.path.join(SRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    noise = "is not a recognized feature for this target"
    err = "\n".join(l for l in (r.stdout + r.stderr).splitlines() if noise not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{err}")
    return obj


def build(verbose=True):
    os.makedirs(OUT_DIR, exist_ok=True)
    with ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        objs = list(ex.map(_compile, SOURCES))
    tmp = LIB + ".tmp"
    r = subprocess.run([HIPCC, "-shared", f"--offload-arch={ARCH}", "-o", tmp, *objs],
                       capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stdout + r.stderr)
    os.replace(tmp, LIB)
    if verbose:
        print(f"built {LIB}")
    return LIB


if __name__ == "__main__":
    build()
    sys.exit(0)
