"""Build libgts.so for gfx950 in-tree.

The host half (extraction, packing, layout) is plain C++ built by g++ without
floating-point contraction; the device half is HIP C++ built by hipcc for
gfx950 with packed-FP32 instruction selection disabled: the launch planner,
the SHAP and interaction kernels (one translation unit per dtype and kind, so
they compile in parallel), and the device path extraction built without
floating-point contraction (its output must equal the host's bit for bit).
The objects are linked into ``paper_2010_13972_amd/libgts.so``.

The compiler's per-kernel resource report (registers, private "scratch"
bytes per lane, occupancy) is kept in ``_build/kernel_resources.txt``.
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


KERNEL_UNITS = ["gts_kernels", "gts_shap_f32", "gts_shap_f64", "gts_inter_f32", "gts_inter_f64",
                "gts_prune"]
RESOURCES = os.path.join(BUILD, "kernel_resources.txt")


def _run_capture(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    lines = [l for l in res.stdout.splitlines()
             if "packed-fp32-ops' is not a recognized feature" not in l]
    if res.returncode != 0:
        raise RuntimeError(f"build step failed ({res.returncode}): {' '.join(cmd)}\n" +
                           "\n".join(lines))
    return lines


def build(verbose: bool = False, save_temps: bool = False) -> str:
    os.makedirs(BUILD, exist_ok=True)
    host_obj = os.path.join(BUILD, "gts_host.o")
    host_cmd = ["g++", *HOST_FLAGS, "-I", INCLUDE, "-I", CSRC, "-c",
                os.path.join(CSRC, "gts_host.cpp"), "-o", host_obj]
    dev_objs, dev_cmds = [], []
    for unit in KERNEL_UNITS:
        obj = os.path.join(BUILD, unit + ".o")
        cmd = ["hipcc", *HIP_FLAGS, "-I", INCLUDE, "-I", CSRC, "-c",
               os.path.join(CSRC, unit + ".hip"), "-o", obj,
               "-Rpass-analysis=kernel-resource-usage"]
        if save_temps:
            cmd += ["-save-temps=obj"]
        dev_objs.append(obj)
        dev_cmds.append(cmd)
    ext_obj = os.path.join(BUILD, "gts_extract.o")
    ext_cmd = ["hipcc", *EXTRACT_FLAGS, "-I", INCLUDE, "-I", CSRC, "-c",
               os.path.join(CSRC, "gts_extract.hip"), "-o", ext_obj,
               "-Rpass-analysis=kernel-resource-usage"]
    cmds = [host_cmd, ext_cmd] + dev_cmds
    with ThreadPoolExecutor(min(len(cmds), os.cpu_count() or 4)) as ex:
        outs = list(ex.map(lambda c: _run_capture(c, verbose), cmds))
    # kernel-resource remarks of the device units, one line per kernel
    report = []
    for lines in outs[1:]:
        cur = {}
        for l in lines:
            if "remark:" not in l:
                continue
            text = l.split("remark:", 1)[1].split("[-Rpass", 1)[0].strip()
            if text.startswith("Function Name:"):
                if cur:
                    report.append(cur)
                cur = {"name": text.split(":", 1)[1].strip()}
            elif ":" in text and cur:
                k, v = text.split(":", 1)
                cur[k.strip()] = v.strip()
        if cur:
            report.append(cur)
    with open(RESOURCES, "w") as f:
        for r in report:
            f.write("\t".join(f"{k}={v}" for k, v in r.items()) + "\n")
    tmp = LIB + ".tmp"
    _run(["hipcc", "--offload-arch=" + ARCH, "-shared", "-fPIC", host_obj, *dev_objs, ext_obj,
          "-o", tmp], verbose)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv, save_temps="--save-temps" in sys.argv))
