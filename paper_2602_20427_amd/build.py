"""Build libgaus.so (the gfx950 HIP library behind include/gaus.h) in-tree."""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libgaus.so")
MICROBENCH = os.path.join(PKG, "gaus_microbench")
SOURCES = ["gaus_host.cpp", "gaus_kernels.hip", "gaus_step.hip", "gaus_poly.hip", "gaus_laplace.hip"]
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

# Packed-FP32 instructions are disabled for device code (they are not needed:
# the kernels are scalar fp32 and the fused multiply-adds issue at full rate).
DEVICE_FLAGS = ["--offload-arch=gfx950", "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _compile(src: str, verbose: bool) -> str:
    path = os.path.join(CSRC, src)
    obj = os.path.join(CSRC, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, "-x", "hip", *DEVICE_FLAGS, "-O3", "-std=c++17", "-fPIC", "-Wall",
           "-I", os.path.join(ROOT, "include"), "-I", CSRC, "-c", path, "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    out = "\n".join(l for l in (r.stdout + r.stderr).splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{out}")
    if verbose and out.strip():
        print(out)
    return obj


def build(verbose: bool = False) -> str:
    """Compile every source for gfx950 and link libgaus.so (always rebuilds)."""
    with ThreadPoolExecutor(max_workers=len(SOURCES)) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose), SOURCES))
    tmp = LIB + ".tmp"
    cmd = [HIPCC, *DEVICE_FLAGS, "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}{r.stderr}")
    os.replace(tmp, LIB)
    for o in objs:
        os.remove(o)
    # unit-rate microbenchmark (standalone executable)
    cmd = [HIPCC, *DEVICE_FLAGS, "-O3", "-std=c++17", "-o", MICROBENCH + ".tmp",
           os.path.join(CSRC, "gaus_microbench.hip")]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"microbenchmark build failed:\n{r.stdout}{r.stderr}")
    os.replace(MICROBENCH + ".tmp", MICROBENCH)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
