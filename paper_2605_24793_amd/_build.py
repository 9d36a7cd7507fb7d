"""Builds libcospec.so (the HIP kernels and the C ABI) in-tree for gfx950."""
from __future__ import annotations

import hashlib
import os
import shutil
import subprocess

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(PKG, "libcospec.so")
SOURCES = ["cospec_api.hip", "reduce.hip", "sample.hip", "head.hip", "scan.hip", "sps.hip", "attention.hip"]
HEADERS = sorted(os.path.join(CSRC, f) for f in os.listdir(CSRC) if f.endswith(".h")) + \
    [os.path.join(INCLUDE, "cospec.h")]


def hipcc() -> str:
    for cand in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if cand and os.path.exists(cand):
            return cand
    raise RuntimeError("hipcc not found (ROCm is required to build libcospec.so)")


def source_files() -> list:
    """Every file the library is built from, in a fixed order: the HIP sources, then
    the headers sorted by path."""
    return [os.path.join(CSRC, s) for s in SOURCES] + HEADERS


def source_hash() -> str:
    """Build id of the current sources: the first 32 hex digits of the SHA-256 of their
    concatenation in source_files() order (the Makefile computes the same)."""
    h = hashlib.sha256()
    for p in source_files():
        with open(p, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:32]


def flags() -> list:
    return ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
            # no packed fp32 VALU instructions anywhere in the device code
            "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
            "-Wall", "-Wno-unused-result", "-I", INCLUDE,
            f"-DCOSPEC_BUILD_ID=\"{source_hash()}\""]


def build(verbose: bool = False) -> str:
    """Compile every HIP source into one shared library; returns its path."""
    tmp = LIB + ".tmp"
    cmd = [hipcc()] + flags() + ["-o", tmp] + [os.path.join(CSRC, s) for s in SOURCES]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + " ".join(cmd) + "\n" + r.stdout + r.stderr)
    if verbose:
        print(" ".join(cmd))
        noise = "is not a recognized feature for this target"
        print("\n".join(l for l in (r.stdout + r.stderr).splitlines() if noise not in l))
    os.replace(tmp, LIB)
    return LIB


def stale() -> bool:
    """True when the library is missing or older than a source or header."""
    if not os.path.exists(LIB):
        return True
    t = os.path.getmtime(LIB)
    return any(os.path.getmtime(p) > t for p in source_files())


if __name__ == "__main__":
    print(build(verbose=True))
