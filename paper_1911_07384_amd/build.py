"""Build libfp16train.so (HIP, gfx950) in-tree with hipcc.

Each .hip source is compiled to an object under ``_build/`` (in parallel),
then linked into ``paper_1911_07384_amd/libfp16train.so``.
"""

from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(HERE, "libfp16train.so")

SOURCES = ["api.hip", "sgd.hip", "bn.hip", "conv_igemm.hip", "conv_wgrad.hip", "conv_f16chain.hip", "layout.hip",
           "pool.hip", "loss.hip", "noalloc.hip"]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
FLAGS = [
    f"--offload-arch={ARCH}",
    "-O3",
    "-std=c++17",
    "-fPIC",
    # every floating-point fusion in this library is an explicit fma
    "-ffp-contract=off",
    # no packed float32 instructions (v_pk_*_f32) anywhere in the device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall",
    "-Wno-unused-function",
]


def _compile(src: str, verbose: bool) -> str:
    obj = os.path.join(BUILD, os.path.splitext(src)[0] + ".o")
    cmd = [HIPCC, *FLAGS, "-c", os.path.join(CSRC, src), "-o", obj]
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
    # hipcc's host pass does not know the packed-fp32 target feature and says so;
    # anything else it prints is shown
    noise = ("packed-fp32-ops", "is not a recognized feature")
    lines = [l for l in (r.stdout + r.stderr).splitlines() if l.strip() and not any(n in l for n in noise)]
    if lines and verbose:
        print("\n".join(lines), flush=True)
    return obj


def build(verbose: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    with cf.ThreadPoolExecutor(max_workers=min(8, len(SOURCES))) as ex:
        objs = list(ex.map(lambda s: _compile(s, verbose), SOURCES))
    # A kernel whose host-side stub was not emitted links fine but fails to
    # load; catch it here (nm lists such stubs as undefined, "U").
    for obj in objs:
        r = subprocess.run(["nm", obj], capture_output=True, text=True, check=True)
        missing = [l.split()[-1] for l in r.stdout.splitlines()
                   if l.split()[0] == "U" and "__device_stub__" in l]
        if missing:
            raise RuntimeError(f"{obj}: kernel stubs not emitted: {missing}")
    tmp = LIB + ".tmp"
    cmd = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
