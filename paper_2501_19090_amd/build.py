"""Compile libpifa.so (hand-written HIP for gfx950) in-tree with hipcc.

    python -m paper_2501_19090_amd.build
"""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libpifa.so")
ARCH = "gfx950"

# Packed fp32 instructions stay off: only scalar / plain vector fp32 code.
HIPCC_FLAGS = [
    "--offload-arch=" + ARCH, "-O3", "-std=c++17", "-fPIC", "-shared",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wall", "-Wno-unused-result",
]


def sources():
    return [os.path.join(CSRC, "pifa.hip")]


def source_digest() -> str:
    """sha256 over the kernel and ABI sources (identifies a kernel version)."""
    import hashlib
    h = hashlib.sha256()
    files = sorted(f for f in os.listdir(CSRC) if f.endswith((".hip", ".hpp")))
    for f in files + ["../../include/pifa.h"]:
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(f.encode())
            h.update(fh.read())
    return h.hexdigest()[:16]


# The headers that hold the forward pass's kernels (the prefill GEMM with its
# epilogues and the decode weight streams); counters taken on one version of
# them stay valid while these files are unchanged.
FORWARD_KERNEL_SOURCES = ("common.hpp", "layout.hpp", "epilogue.hpp", "gemm_mfma.hpp", "gemv_skinny.hpp",
                          "prepack.hpp")


def forward_kernel_digest() -> str:
    """sha256 over the forward kernels' headers (identifies their version)."""
    import hashlib
    h = hashlib.sha256()
    for f in FORWARD_KERNEL_SOURCES:
        with open(os.path.join(CSRC, f), "rb") as fh:
            h.update(f.encode())
            h.update(fh.read())
    return h.hexdigest()[:16]


def build(verbose: bool = False) -> str:
    """Always recompile (this is the build check); returns the library path."""
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    tmp = LIB + ".tmp%d" % os.getpid()
    cmd = [hipcc] + HIPCC_FLAGS + ["-I", os.path.join(ROOT, "include"), "-o", tmp] + sources()
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in res.stdout.splitlines() if "packed-fp32-ops" not in l)
    if res.returncode != 0:
        if os.path.exists(tmp):
            os.remove(tmp)
        raise RuntimeError("hipcc failed:\n" + out)
    if verbose and out.strip():
        print(out)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
