"""Build the HIP library libbase.so in-tree for gfx950.

Every source is compiled by hipcc with:
  -O3 -std=c++17 -fPIC --offload-arch=gfx950
  -ffp-contract=off     (no implicit FMA: the scoring path's fp32 order is
                         fixed and uses fmaf() only where it says so)
  -Xclang -target-feature -Xclang -packed-fp32-ops
                        (no packed fp32 VALU instructions)
The default HIP settings keep fp32 division and square root correctly
rounded and fp32 denormals enabled; nothing here changes them.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OUT_DIR = os.path.join(HERE, "_lib")
LIB = os.path.join(OUT_DIR, "libbase.so")
PROBE_LIB = os.path.join(OUT_DIR, "libbase_probe.so")   # bench's streaming-read probe
CALIB_LIB = os.path.join(OUT_DIR, "libbase_calib.so")   # predictor fit (links rocSOLVER)
SOURCES = ["api.hip", "scores.hip", "plan.hip", "ffn.hip",
           "pack.hip", "calib.hip"]
ARCH = os.environ.get("BASE_OFFLOAD_ARCH", "gfx950")

FLAGS = ["-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}",
         "-ffp-contract=off",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
         "-Wno-unused-command-line-argument"]


def _hipcc():
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", "hipcc"):
        if c and (os.path.sep not in c or os.path.exists(c)):
            return c
    raise RuntimeError("hipcc not found")


def _link(objs, out, libs=()):
    tmp = out + ".tmp%d" % os.getpid()
    cmd = [_hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp, *libs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stderr}")
    os.replace(tmp, out)


def build(verbose: bool = False) -> str:
    """Compile every source, link libbase.so and the probe library (always
    rebuilds)."""
    os.makedirs(OUT_DIR, exist_ok=True)
    hipcc = _hipcc()
    objs = []

    def compile_one(src):
        obj = os.path.join(OUT_DIR, src.replace(".hip", ".o"))
        cmd = [hipcc, *FLAGS, "-c", os.path.join(CSRC, src), "-o", obj]
        r = subprocess.run(cmd, capture_output=True, text=True)
        if r.returncode != 0:
            raise RuntimeError(f"hipcc failed on {src}:\n{r.stderr}")
        if verbose and r.stderr.strip():
            print(r.stderr, file=sys.stderr)
        return obj

    with cf.ThreadPoolExecutor(min(8, len(SOURCES) + 2)) as ex:
        objs = list(ex.map(compile_one, SOURCES + ["probe.hip", "calib_fit.hip"]))
    _link(objs[:-2], LIB)
    _link(objs[-2:-1], PROBE_LIB)
    _link(objs[-1:], CALIB_LIB, ["-lrocsolver", "-lrocblas"])
    for o in objs:
        os.remove(o)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
