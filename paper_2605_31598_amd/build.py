"""Build the gfx950 shared libraries in-tree with hipcc.

* ``paper_2605_31598_amd/libstatekv.so``: the frame-step library (C ABI of include/statekv.h).
* ``workloads/libskvgen.so``: the device input generator used to fill benchmark inputs.

Every HIP translation unit is compiled with packed-fp32 instructions disabled.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

CSRC = os.path.join(PKG, "csrc")
SOURCES = ["statekv.hip", "attn_mfma.hip", "attn_full.hip", "attn_decode.hip", "attn_simple.hip", "refresh.hip",
           "rope_keys.hip", "plan.cpp"]
LIB = os.path.join(PKG, "libstatekv.so")
GEN_SRC = os.path.join(ROOT, "workloads", "csrc", "skv_gen.hip")
GEN_LIB = os.path.join(ROOT, "workloads", "libskvgen.so")

FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-command-line-argument",
    f"-I{os.path.join(ROOT, 'include')}",
]


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in r.stdout.splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{out}")
    return out


def build(verbose: bool = False) -> list:
    obj_dir = os.path.join(PKG, "_build")
    os.makedirs(obj_dir, exist_ok=True)
    objs = [os.path.join(obj_dir, os.path.splitext(s)[0] + ".o") for s in SOURCES]
    jobs = [[HIPCC, *FLAGS, "-c", os.path.join(CSRC, s), "-o", o] for s, o in zip(SOURCES, objs)]
    with cf.ThreadPoolExecutor(max_workers=min(len(jobs) + 1, 8)) as ex:
        futs = [ex.submit(_run, j) for j in jobs]
        futs.append(ex.submit(_run, [HIPCC, *FLAGS, "-shared", GEN_SRC, "-o", GEN_LIB + ".tmp"]))
        for f in futs:
            out = f.result()
            if verbose and out.strip():
                print(out)
    _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", LIB + ".tmp"])
    os.replace(LIB + ".tmp", LIB)
    os.replace(GEN_LIB + ".tmp", GEN_LIB)
    return [LIB, GEN_LIB]


if __name__ == "__main__":
    for p in build(verbose="-v" in sys.argv):
        print(p)
