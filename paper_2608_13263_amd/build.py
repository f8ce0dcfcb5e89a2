"""Build libvtoken.so (the HIP kernels and the C ABI of include/vtoken.h) for gfx950.

    python -m paper_2608_13263_amd.build

Compiles in-tree with hipcc; the library lands next to this file, where the binding loads it.
Packed-FP32 instructions are disabled for all device code. The SHA-256 of the sources
(`source_sha256()`: every file of csrc/ and include/vtoken.h) is compiled in and returned by
vtoken_build_id(), so a loaded library can be tied to the tree it was built from.
"""
from __future__ import annotations

import hashlib
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
LIB_PATH = os.path.join(HERE, "libvtoken.so")
CSRC = os.path.join(HERE, "csrc")
SOURCES = [os.path.join(CSRC, f)
           for f in ("vtoken_abi.hip", "vtoken_kernels.hip", "vtoken_copy.hip",
                     "vtoken_attention.hip", "vtoken_planner.hip", "vtoken_layout.hip")]
HEADERS = [os.path.join(ROOT, "include", "vtoken.h"), os.path.join(CSRC, "vtoken_internal.h")]
ARCH = "gfx950"


def source_files():
    """Every file the library is built from: csrc/ (all of it) and the public header."""
    files = [os.path.join(CSRC, f) for f in os.listdir(CSRC)
             if f.endswith((".hip", ".h")) and os.path.isfile(os.path.join(CSRC, f))]
    return sorted(files + [os.path.join(ROOT, "include", "vtoken.h")])


def source_sha256() -> str:
    """SHA-256 over the source files in sorted order of their paths relative to the repository
    root: for each, the path, a NUL byte, the contents, a NUL byte."""
    h = hashlib.sha256()
    for path in source_files():
        h.update(os.path.relpath(path, ROOT).encode() + b"\0")
        with open(path, "rb") as f:
            h.update(f.read())
        h.update(b"\0")
    return h.hexdigest()


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found; install ROCm or set HIPCC")


def command(out_path: str, sources, defines=()):
    return [hipcc(), f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared",
            "-Wall", "-Wno-unused-function",
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-I", os.path.join(ROOT, "include"), "-I", CSRC,
            *(f"-D{d}" for d in defines), *sources, "-o", out_path]


def build_id_defines(sha: str):
    # four 64-bit words of the hash as numeric macros (no quoting through the compiler driver)
    return [f"VTOKEN_SRC_SHA{i}=0x{sha[16 * i:16 * (i + 1)]}ULL" for i in range(4)]


def build(verbose: bool = False) -> str:
    """Compile libvtoken.so (always, even if it exists); returns its path."""
    return build_one(LIB_PATH, SOURCES, build_id_defines(source_sha256()), verbose)


def build_one(lib_path: str, sources, defines=(), verbose: bool = False) -> str:
    """Compile `sources` into `lib_path`, installed atomically."""
    tmp = lib_path + ".tmp"
    cmd = command(tmp, sources, defines)
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
