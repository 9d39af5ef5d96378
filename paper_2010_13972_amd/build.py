"""Build libgts.so for gfx950 in-tree.

The host half (extraction, packing, layout) is plain C++ built by g++ without
floating-point contraction; the device half is HIP C++ built by hipcc for
gfx950 with packed-FP32 instruction selection disabled: the SHAP kernels, and
the device path extraction built without floating-point contraction (its
output must equal the host's bit for bit).  The objects are linked into
``paper_2010_13972_amd/libgts.so``.
"""
from __future__ import annotations

import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(HERE, "_build")
LIB = os.path.join(HERE, "libgts.so")
ARCH = "gfx950"

HOST_FLAGS = ["-O2", "-std=c++17", "-fPIC", "-ffp-contract=off", "-Wall", "-Wextra",
              "-Wno-unused-parameter"]
HIP_COMMON = ["--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC",
              "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
HIP_FLAGS = HIP_COMMON + ["-ffp-contract=fast", "-munsafe-fp-atomics"]
EXTRACT_FLAGS = HIP_COMMON + ["-ffp-contract=off"]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in res.stdout.splitlines()
                    if "packed-fp32-ops' is not a recognized feature" not in l)
    if res.returncode != 0:
        raise RuntimeError(f"build step failed ({res.returncode}): {' '.join(cmd)}\n{out}")
    if verbose and out.strip():
        print(out)


def build(verbose: bool = False, save_temps: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    host_obj = os.path.join(BUILD, "gts_host.o")
    dev_obj = os.path.join(BUILD, "gts_kernels.o")
    host_cmd = ["g++", *HOST_FLAGS, "-I", INCLUDE, "-I", CSRC, "-c",
                os.path.join(CSRC, "gts_host.cpp"), "-o", host_obj]
    dev_cmd = ["hipcc", *HIP_FLAGS, "-I", INCLUDE, "-I", CSRC, "-c",
               os.path.join(CSRC, "gts_kernels.hip"), "-o", dev_obj]
    ext_obj = os.path.join(BUILD, "gts_extract.o")
    ext_cmd = ["hipcc", *EXTRACT_FLAGS, "-I", INCLUDE, "-I", CSRC, "-c",
               os.path.join(CSRC, "gts_extract.hip"), "-o", ext_obj]
    if save_temps:
        dev_cmd += ["-save-temps=obj"]
    with ThreadPoolExecutor(3) as ex:
        futs = [ex.submit(_run, c, verbose) for c in (host_cmd, dev_cmd, ext_cmd)]
        for f in futs:
            f.result()
    tmp = LIB + ".tmp"
    _run(["hipcc", "--offload-arch=" + ARCH, "-shared", "-fPIC", host_obj, dev_obj, ext_obj,
          "-o", tmp], verbose)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv, save_temps="--save-temps" in sys.argv))
