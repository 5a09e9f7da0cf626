"""Builds libsherry.so (HIP for gfx950) in-tree with hipcc.

Every source under csrc/ is compiled to an object in _build/ and linked into
paper_2601_07892_amd/libsherry.so.  Flags:
  * --offload-arch=gfx950 only (no other targets, no host fallback);
  * packed-fp32 instructions disabled (-packed-fp32-ops);
  * correctly rounded fp32 division and no denormal flushing, so the
    activation quantizer's fp32 decisions are IEEE ones.
"""
from __future__ import annotations

import concurrent.futures as cf
import glob
import os
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(PKG, "libsherry.so")

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
FLAGS = [
    "--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-fhip-fp32-correctly-rounded-divide-sqrt", "-fno-gpu-flush-denormals-to-zero",
    "-ffp-contract=off", "-Wall", "-Wno-unused-function",
    "-I" + os.path.join(ROOT, "include"),
]


def _compile(src: str) -> str:
    obj = os.path.join(BUILD, os.path.basename(src) + ".o")
    subprocess.run([HIPCC, *FLAGS, "-c", src, "-o", obj], check=True,
                   stdout=subprocess.PIPE, stderr=subprocess.STDOUT)
    return obj


def build(save_temps: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    srcs = sorted(glob.glob(os.path.join(CSRC, "*.hip")))
    if save_temps:
        FLAGS.append("-save-temps=obj")
    try:
        with cf.ThreadPoolExecutor(max_workers=min(8, len(srcs))) as ex:
            objs = list(ex.map(_compile, srcs))
    except subprocess.CalledProcessError as e:  # show the compiler output
        raise RuntimeError("hipcc failed:\n" + e.stdout.decode(errors="replace")) from None
    tmp = LIB + ".tmp%d" % os.getpid()
    r = subprocess.run([HIPCC, "--offload-arch=" + ARCH, "-shared", "-fPIC", *objs, "-o", tmp,
                        "-lpthread"], stdout=subprocess.PIPE, stderr=subprocess.STDOUT)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n" + r.stdout.decode(errors="replace"))
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build())
