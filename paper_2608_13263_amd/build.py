"""Build libvtoken.so (the HIP kernels and the C ABI of include/vtoken.h) and
libvtoken_probe.so (the memory-system streaming probes of `bench.py --mode stream`) for gfx950.

    python -m paper_2608_13263_amd.build

Compiles in-tree with hipcc; the libraries land next to this file, where the binding and the
benchmark load them. Packed-FP32 instructions are disabled for all device code.
"""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB_PATH = os.path.join(HERE, "libvtoken.so")
SOURCES = [os.path.join(HERE, "csrc", f)
           for f in ("vtoken_abi.hip", "vtoken_kernels.hip", "vtoken_attention.hip",
                     "vtoken_planner.hip", "vtoken_layout.hip")]
HEADERS = [os.path.join(ROOT, "include", "vtoken.h"),
           os.path.join(HERE, "csrc", "vtoken_internal.h")]
PROBE_LIB_PATH = os.path.join(HERE, "libvtoken_probe.so")
PROBE_SOURCES = [os.path.join(HERE, "csrc", "vtoken_stream_probe.hip")]
ARCH = "gfx950"


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found; install ROCm or set HIPCC")


def command(out_path: str, sources=None):
    return [hipcc(), f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared",
            "-Wall", "-Wno-unused-function",
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-I", os.path.join(ROOT, "include"), "-I", os.path.join(HERE, "csrc"),
            *(sources or SOURCES), "-o", out_path]


def build(verbose: bool = False) -> str:
    """Compile both libraries (always, even if they exist); returns libvtoken.so's path."""
    build_one(PROBE_LIB_PATH, PROBE_SOURCES, verbose)
    return build_one(LIB_PATH, SOURCES, verbose)


def build_one(lib_path: str, sources, verbose: bool = False) -> str:
    """Compile `sources` into `lib_path`, installed atomically."""
    tmp = lib_path + ".tmp"
    cmd = command(tmp, sources)
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError(f"hipcc failed with exit code {res.returncode}")
    if verbose and res.stderr.strip():
        # hipcc's host pass warns that it does not know the packed-fp32 feature: harmless
        lines = [ln for ln in res.stderr.splitlines() if "packed-fp32-ops" not in ln]
        if any(ln.strip() for ln in lines):
            sys.stderr.write("\n".join(lines) + "\n")
    os.replace(tmp, lib_path)
    return lib_path


if __name__ == "__main__":
    print(build(verbose=True))
