"""Builds libchunk.so (HIP kernels for gfx950 + host core) in-tree.

    python -m paper_2606_11169_amd.build        # or __graft_entry__.build()

Every call recompiles: the host core with the host C++ compiler, each .hip
file with hipcc for gfx950 (in parallel), then links one shared library at
paper_2606_11169_amd/_lib/libchunk.so.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
OUT_DIR = os.path.join(HERE, "_lib")
OBJ_DIR = os.path.join(OUT_DIR, "obj")
LIB = os.path.join(OUT_DIR, "libchunk.so")

ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
HIPCC = os.path.join(ROCM, "bin", "hipcc")
ARCH = "gfx950"

HIP_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", f"-I{INCLUDE}", f"-I{CSRC}",
    # no packed-fp32 instructions anywhere in the device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-fhip-fp32-correctly-rounded-divide-sqrt",
    "-Wno-unused-result",
]
# kernels whose results are defined operation by operation (bit-exact paths)
NO_CONTRACT = {"k_optim.hip"}
# per-file code generation options
EXTRA_FLAGS = {
    # keep MFMA results in VGPRs: the attention kernels apply the softmax to
    # them with vector instructions, and accumulation-register copies cost more
    # than they save
    "k_attn.hip": ["-mllvm", "-amdgpu-mfma-vgpr-form"],
}


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in r.stdout.splitlines() if "not a recognized feature" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{out}")
    return out


def build(verbose: bool = False) -> str:
    if not os.path.exists(HIPCC):
        raise RuntimeError(f"hipcc not found at {HIPCC}")
    os.makedirs(OBJ_DIR, exist_ok=True)
    jobs = []
    cxx = shutil.which("g++") or "c++"
    host_obj = os.path.join(OBJ_DIR, "host_core.o")
    jobs.append([cxx, "-std=c++17", "-O2", "-fPIC", "-Wall", f"-I{INCLUDE}", "-c",
                 os.path.join(CSRC, "host_core.cpp"), "-o", host_obj])
    objs = [host_obj]
    for f in sorted(os.listdir(CSRC)):
        if not f.endswith(".hip"):
            continue
        o = os.path.join(OBJ_DIR, f[:-4] + ".o")
        flags = list(HIP_FLAGS)
        if f in NO_CONTRACT:
            flags.append("-ffp-contract=off")
        flags.extend(EXTRA_FLAGS.get(f, []))
        jobs.append([HIPCC, *flags, "-c", os.path.join(CSRC, f), "-o", o])
        objs.append(o)
    workers = min(len(jobs), max(1, min(8, os.cpu_count() or 1)))
    with cf.ThreadPoolExecutor(workers) as ex:
        outs = list(ex.map(_run, jobs))
    tmp = LIB + ".tmp"
    link = [HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp]
    outs.append(_run(link))
    os.replace(tmp, LIB)
    if verbose:
        for o in outs:
            if o.strip():
                print(o)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
