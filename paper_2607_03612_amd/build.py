"""Builds libsaf3r.so (the gfx950 HIP kernels + the C ABI) in the package directory.

Usage: python -m paper_2607_03612_amd.build [--verbose]
"""
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
LIB = os.path.join(PKG, "libsaf3r.so")
SOURCES = ["api.cpp", "pool.hip", "select.hip", "attn.hip", "cosine.hip", "nmse.hip"]
ARCH = "gfx950"


def hipcc() -> str:
    path = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(path):
        raise RuntimeError("hipcc not found: the HIP library cannot be built")
    return path


def command(out: str = LIB, extra=()) -> list:
    return [
        hipcc(), f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared",
        # packed fp32 VALU ops are kept out of the generated code
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        "-Wno-unused-command-line-argument",
        "-I", os.path.join(ROOT, "include"),
        *extra,
        *[os.path.join(CSRC, s) for s in SOURCES],
        "-o", out,
    ]


def device_asm(source: str, out: str) -> str:
    """AMD assembly of one kernel source for gfx950 (device code only, the
    same flags as the library), written to `out`."""
    cmd = [
        hipcc(), f"--offload-arch={ARCH}", "-O3", "-std=c++17",
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        "-Wno-unused-command-line-argument",
        "-I", os.path.join(ROOT, "include"), "-I", CSRC,
        "--cuda-device-only", "-S", os.path.join(CSRC, source), "-o", out,
    ]
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError(f"hipcc -S {source} failed with status {res.returncode}")
    return out


def build(verbose: bool = False) -> str:
    """Compile every source for gfx950 into the package's libsaf3r.so."""
    tmp = LIB + ".tmp"
    cmd = command(tmp)
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    if res.returncode != 0:
        sys.stderr.write(res.stdout + res.stderr)
        raise RuntimeError(f"hipcc failed with status {res.returncode}")
    os.replace(tmp, LIB)
    return LIB


if __name__ == "__main__":
    print(build(verbose="--verbose" in sys.argv))
