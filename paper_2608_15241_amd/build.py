"""Build liblocal.so (the C-ABI library) from csrc/ with hipcc for gfx950.

    python -m paper_2608_15241_amd.build

The library is built in-tree, next to this file, and always from scratch.
"""
from __future__ import annotations

import glob
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
LIB = os.path.join(HERE, "liblocal.so")
ARCH = "gfx950"

HIPCC_FLAGS = [
    "-O3", "-std=c++17", "-fPIC", "-shared",
    "--offload-arch=" + ARCH,
    # The runtime bundled with PyTorch loads code objects of version 5.
    "-mcode-object-version=5",
    # Keep packed-fp32 instructions out of the device code.
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-command-line-argument",
]


def sources():
    """The HIP kernels and the C ABI (csrc/*.hip)."""
    return sorted(glob.glob(os.path.join(HERE, "csrc", "*.hip")))


def host_sources():
    """Host-only C++ (the KV manager, csrc/*.cpp), compiled with g++."""
    return sorted(glob.glob(os.path.join(HERE, "csrc", "*.cpp")))


def build(verbose: bool = False) -> str:
    hipcc = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
    tmp = LIB + ".tmp%d" % os.getpid()
    objs = []
    for src in host_sources():
        obj = "%s.%d.o" % (src[:-4], os.getpid())
        cmd = ["g++", "-O2", "-std=c++17", "-fPIC", "-Wall", "-c", src, "-o", obj]
        if verbose:
            print(" ".join(cmd), flush=True)
        res = subprocess.run(cmd, capture_output=True, text=True)
        if res.returncode != 0:
            raise RuntimeError("g++ failed (%d):\n%s" % (res.returncode, res.stderr))
        objs.append(obj)
    # the objects go straight to the linker (hipcc would read them as HIP)
    cmd = [hipcc] + HIPCC_FLAGS + sources() + ["-Wl," + o for o in objs] + ["-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    try:
        res = subprocess.run(cmd, capture_output=True, text=True)
    finally:
        for obj in objs:
            if os.path.exists(obj):
                os.remove(obj)
    # hipcc's host pass warns that it does not know the packed-fp32 feature.
    err = "\n".join(l for l in res.stderr.splitlines()
                    if "packed-fp32-ops" not in l or "error" in l)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed (%d):\n%s" % (res.returncode, err))
    if verbose and err.strip():
        print(err, file=sys.stderr)
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose=True))
