"""Build libsplash_attn.so in-tree with hipcc for gfx950.

Usage: python -m paper_2609_37626_amd.build
"""
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIB = os.path.join(HERE, "libsplash_attn.so")
SOURCES = ["api.cpp", "kernels.hip", "dop.hip"]
# measurement helpers for the benchmark, a library of their own
CALIB_LIB = os.path.join(HERE, "libsplash_calib.so")
CALIB_SOURCES = ["calib.hip"]

HIPCC_FLAGS = [
    "--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-Wall", "-Wno-unused-command-line-argument",
    # keep hipcc from emitting packed fp32 arithmetic
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", INCLUDE, "-I", CSRC,
]


def hipcc() -> str:
    exe = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(exe):
        raise RuntimeError("hipcc not found")
    return exe


def build(verbose: bool = False) -> str:
    """Compile libsplash_attn.so and libsplash_calib.so (always rebuilds)."""
    _compile(CALIB_SOURCES, CALIB_LIB, verbose)
    return _compile(SOURCES, LIB, verbose)


def _compile(sources, lib, verbose: bool) -> str:
    tmp = lib + ".tmp"
    cmd = [hipcc()] + HIPCC_FLAGS + [os.path.join(CSRC, s) for s in sources] + ["-o", tmp]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    noise = ("packed-fp32-ops", "warning: feature flag", "1 warning generated")
    msgs = [l for l in (res.stdout + res.stderr).splitlines() if not any(n in l for n in noise)]
    if res.returncode != 0:
        raise RuntimeError("hipcc failed:\n" + "\n".join(msgs))
    if verbose and msgs:
        print("\n".join(msgs))
    os.replace(tmp, lib)
    return lib


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
