"""Build libgmlp.so (HIP, gfx950) in-tree with hipcc.

    python -m paper_2606_26344_amd.build

The library is compiled for gfx950 only, with every warning an error.
Packed fp32 instructions are disabled for all device code
(-packed-fp32-ops).
"""
from __future__ import annotations

import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
LIBRARY = os.path.join(PKG, "libgmlp.so")
SOURCES = [os.path.join(CSRC, "gmlp.hip")]
# A measuring program beside the library (not part of it): the board's
# sustained bf16 matrix-core rate, which bench.py reports as context.
MFMA_CEILING = os.path.join(PKG, "mfma_ceiling")
MFMA_CEILING_SOURCE = os.path.join(CSRC, "mfma_ceiling.hip")
HEADERS = [os.path.join(CSRC, f) for f in sorted(os.listdir(CSRC)) if f.endswith(".hpp")] + [
    os.path.join(INCLUDE, h) for h in ("gmlp.h", "softmax_matmul.h")]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    "--offload-arch=gfx950",
    "-O3",
    "-std=c++20",
    "-shared",
    "-fPIC",
    "-Wall",
    "-Wextra",
    "-Werror",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-I", INCLUDE,
    "-I", CSRC,
]


def _compile(out, flags, sources, verbose):
    tmp = out + ".tmp%d" % os.getpid()
    cmd = [HIPCC, *flags, "-o", tmp, *sources]
    if verbose:
        print(" ".join(cmd), flush=True)
    res = subprocess.run(cmd, capture_output=True, text=True)
    noise = "warning: unknown target feature"
    msgs = [ln for ln in (res.stdout + res.stderr).splitlines() if ln.strip()]
    shown = [ln for ln in msgs if noise not in ln and "packed-fp32-ops" not in ln]
    if shown and (verbose or res.returncode != 0):
        print("\n".join(shown), file=sys.stderr)
    if res.returncode != 0:
        raise RuntimeError("hipcc failed with exit code %d" % res.returncode)
    os.replace(tmp, out)


def build(verbose: bool = False, extra_flags=()) -> str:
    """Compile libgmlp.so (and the mfma_ceiling program) next to this file;
    returns the library's path."""
    _compile(LIBRARY, [*FLAGS, *extra_flags], SOURCES, verbose)
    exe_flags = [f for f in FLAGS if f not in ("-shared", "-fPIC")]
    _compile(MFMA_CEILING, exe_flags, [MFMA_CEILING_SOURCE], verbose)
    return LIBRARY


def is_stale() -> bool:
    if not os.path.exists(LIBRARY) or not os.path.exists(MFMA_CEILING):
        return True
    t = os.path.getmtime(LIBRARY)
    return (any(os.path.getmtime(f) > t for f in SOURCES + HEADERS) or
            os.path.getmtime(MFMA_CEILING_SOURCE) > os.path.getmtime(MFMA_CEILING))


if __name__ == "__main__":
    print(build(verbose=True))
