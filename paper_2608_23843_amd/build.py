"""Builds libpuzzlekv.so (the HIP kernels and the C ABI) in-tree for gfx950."""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libpuzzlekv.so")

SOURCES = ["pkv_kernels.hip", "pkv_host.cpp"]
DEPS = ["pkv_internal.h", "cache_ops.inl", "int4.inl", "compress.inl", "compress_qr.inl", "attention.inl", "attention_mfma.inl", "attention_q4.inl",
        "attention_launch.inl", "global_svd.inl", "bandwidth.inl"]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found: the PuzzleKV library needs the ROCm toolchain")


def flags() -> list[str]:
    return [
        "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC",
        # packed fp32 instructions are left to nobody: the compiler may not form them
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        # the page-claim atomics are issued by one lane whose result is read
        # later; the wave-level atomic rewrite would read it at once, waiting
        # for every load issued before it
        "-mllvm", "-amdgpu-atomic-optimizer-strategy=None",
        # matrix-core accumulators in VGPRs: the decomposition's Gram tiles are
        # short-lived and AGPRs would cost it a wave per SIMD (every other
        # kernel compiles to the same code either way)
        "-mllvm", "-amdgpu-mfma-vgpr-form=1",
        "-Wno-unused-command-line-argument",
        "-I", INCLUDE, "-I", CSRC,
    ]


def build(verbose: bool = False) -> str:
    """Compiles every source (always) and links libpuzzlekv.so next to this file."""
    objs = []
    tmpdir = os.path.join(HERE, "_build")
    os.makedirs(tmpdir, exist_ok=True)
    for src in SOURCES:
        obj = os.path.join(tmpdir, src + ".o")
        cmd = [hipcc()] + flags() + ["-c", os.path.join(CSRC, src), "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        subprocess.check_call(cmd)
        objs.append(obj)
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [hipcc(), "--offload-arch=gfx950", "-shared", "-fPIC", "-o", tmp] + objs
    if verbose:
        print(" ".join(cmd), flush=True)
    subprocess.check_call(cmd)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
