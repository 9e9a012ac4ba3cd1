"""Builds libonexn.so (HIP kernels for gfx950 + host C++) in-tree.

    python -m paper_2105_14713_amd.build

hipcc cross-compiles for gfx950; no GPU is needed to build.
"""
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INC = os.path.join(ROOT, "include")
OUT = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libonexn.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"

# Packed fp32 VALU ops are disabled for all device code (see the kernel notes).
DEVICE_FLAGS = ["-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
HIP_SOURCES = ["onexn_conv.hip", "conv_generic.hip", "conv_pw_tile.hip", "conv_pw_bf16r.hip",
               "conv_pw_bf16s.hip", "conv_kxk.hip", "conv_kxk_fma.hip", "conv_pw_fma.hip", "conv_pw_direct.hip",
               "conv_pw_nhwc.hip",
               "mask_dev.hip", "conv_bwd.hip", "conv_bwd_pw.hip"]
COMMON = ["-O3", "-std=c++17", "-fPIC", "-Wall", "-I" + INC, "-I" + CSRC]


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.run(cmd, check=True)


def build(verbose: bool = False) -> str:
    os.makedirs(OUT, exist_ok=True)
    host_o = os.path.join(OUT, "onexn_host.o")
    jobs = [(["g++"] + COMMON + ["-c", os.path.join(CSRC, "onexn_host.cpp"), "-o", host_o])]
    objs = [host_o]
    for src in HIP_SOURCES:
        obj = os.path.join(OUT, src.replace(".hip", ".o"))
        jobs.append([HIPCC, "--offload-arch=" + ARCH] + COMMON + DEVICE_FLAGS +
                    ["-c", os.path.join(CSRC, src), "-o", obj])
        objs.append(obj)
    procs = []
    for cmd in jobs:
        if verbose:
            print(" ".join(cmd), flush=True)
        procs.append((cmd, subprocess.Popen(cmd)))
    for cmd, proc in procs:
        if proc.wait() != 0:
            raise subprocess.CalledProcessError(proc.returncode, cmd)
    tmp = LIB + ".tmp"
    _run([HIPCC, "--offload-arch=" + ARCH, "-shared", "-fPIC"] + objs + ["-o", tmp], verbose)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
