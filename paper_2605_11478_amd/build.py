"""Build libfibq.so in-tree: host C++ with g++, HIP kernels with hipcc for gfx950.

Usage: ``python -m paper_2605_11478_amd.build`` (or ``build()`` from Python).
Always recompiles; objects go to ``paper_2605_11478_amd/_build/``.
"""
import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
OUT = os.path.join(PKG, "libfibq.so")
BUILD = os.path.join(PKG, "_build")

HOST_SRC = ["api.cpp", "host_builder.cpp"]
HIP_SRC = ["codec_kernels.hip", "encode_mfma.hip", "encode_mf4.hip", "encode_big.hip", "attn_kernels.hip", "attn_fast.hip", "attn_w4.hip", "attn_k4.hip", "attn_noalloc.hip"]

HIP_FLAGS = [
    "-O3", "-std=c++17", "-fPIC", "--offload-arch=gfx950",
    # no packed fp32 instructions in device code
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-command-line-argument",
    # matrix-core accumulators in ordinary VGPRs (no AGPR copies around them)
    "-mllvm", "-amdgpu-mfma-vgpr-form",
    # work-claiming atomics are issued by one lane; no wave-level rewriting
    "-mllvm", "-amdgpu-atomic-optimizer-strategy=None",
]
HOST_FLAGS = ["-O3", "-std=c++17", "-fPIC", "-Wall", "-Wextra", "-Wno-unused-parameter"]


def _hipcc():
    for c in (shutil.which("hipcc"), "/opt/rocm/bin/hipcc"):
        if c and os.path.exists(c):
            return c
    raise RuntimeError("hipcc not found")


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    if r.returncode != 0:
        raise RuntimeError("build step failed:\n" + " ".join(cmd) + "\n" + r.stdout)
    return r.stdout


def build(verbose=False):
    os.makedirs(BUILD, exist_ok=True)
    hipcc = _hipcc()
    inc = ["-I", INCLUDE, "-I", CSRC]
    jobs = []
    objs = []
    for s in HOST_SRC:
        o = os.path.join(BUILD, s + ".o")
        jobs.append(["g++", *HOST_FLAGS, *inc, "-c", os.path.join(CSRC, s), "-o", o])
        objs.append(o)
    for s in HIP_SRC:
        o = os.path.join(BUILD, s + ".o")
        jobs.append([hipcc, *HIP_FLAGS, *inc, "-c", os.path.join(CSRC, s), "-o", o])
        objs.append(o)
    with ThreadPoolExecutor(max_workers=4) as ex:
        outs = list(ex.map(_run, jobs))
    if verbose:
        for o in outs:
            if o.strip():
                print(o)
    tmp = OUT + ".tmp"
    _run([hipcc, "-shared", "-fPIC", "--offload-arch=gfx950", *objs, "-o", tmp, "-lpthread"])
    os.replace(tmp, OUT)
    return OUT


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
