"""Builds the HIP library of the fused linear + cross-entropy step for gfx950.

    python -m paper_2603_16428_amd.build

compiles csrc/lce_api.hip (which includes the kernels) and csrc/host_adam.cpp (the host optimizer
step) into liblce.so next to this file.
"""
from __future__ import annotations

import os
import subprocess
import sys
import tempfile

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB = os.path.join(HERE, "liblce.so")
KERNEL_SOURCES = [os.path.join(HERE, "csrc", "lce_api.hip")]
HOST_SOURCES = [os.path.join(HERE, "csrc", "host_adam.cpp")]
SOURCES = KERNEL_SOURCES + HOST_SOURCES
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")

FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    # No packed fp32 arithmetic in device code.
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", os.path.join(ROOT, "include"),
]


# Host-only C++ (the optimizer step: function multiversioning and x86 _Float16, which the HIP
# compile of a .cpp would also try to build for the GPU) goes through the host compiler first.
HOSTCXX = os.environ.get("LCE_HOSTCXX", "/opt/rocm/llvm/bin/clang++")
HOST_FLAGS = ["-O3", "-std=c++17", "-fPIC", "-I", os.path.join(ROOT, "include")]


def build(verbose: bool = False) -> str:
    """Compile liblce.so (always) and return its path. Raises on failure."""
    tmp = LIB + ".tmp"
    with tempfile.TemporaryDirectory() as d:
        objs = []
        for src in HOST_SOURCES:
            obj = os.path.join(d, os.path.splitext(os.path.basename(src))[0] + ".o")
            r = subprocess.run([HOSTCXX] + HOST_FLAGS + ["-c", src, "-o", obj], capture_output=True, text=True)
            if r.returncode != 0:
                raise RuntimeError(f"{HOSTCXX} failed on {src}:\n" + r.stdout + r.stderr)
            objs.append(obj)
        # Objects first: hipcc's language flag for the .hip sources applies to the inputs after it.
        cmd = [HIPCC] + FLAGS + objs + KERNEL_SOURCES + ["-pthread", "-o", tmp]
        r = subprocess.run(cmd, capture_output=True, text=True)
    msgs = [ln for ln in (r.stdout + r.stderr).splitlines() if "packed-fp32-ops" not in ln]
    if r.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + "\n".join(msgs))
    if verbose and msgs:
        print("\n".join(msgs), file=sys.stderr)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
