"""Build liblattice.so (gfx950) in-tree with hipcc.

Every library translation unit under ``csrc/`` is compiled in parallel to an
object under ``_build/`` and linked into ``_lib/liblattice.so``.  ``peaks.hip``
(sustained MFMA and HBM rates, a measurement aid) becomes its own executable,
``_lib/peaks``.  The splat unit is
compiled without floating-point contraction: the enclosing-simplex decision
must follow one fixed sequence of individually rounded fp32 operations.
"""
from __future__ import annotations

import os
import subprocess
from concurrent.futures import ThreadPoolExecutor

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
BUILD = os.path.join(PKG, "_build")
LIBDIR = os.path.join(PKG, "_lib")
LIB = os.path.join(LIBDIR, "liblattice.so")
ARCH = "gfx950"

SOURCES = ["lattice.hip", "splat.hip", "neighbors.hip", "conv.hip", "slice.hip", "deform.hip", "deform_bwd.hip",
           "backward.hip", "distribute.hip"]
EXTRA = {"splat.hip": ["-ffp-contract=off"]}
PEAKS_SRC = "peaks.hip"
PEAKS = os.path.join(LIBDIR, "peaks")


def hipcc() -> str:
    rocm = os.environ.get("ROCM_PATH", "/opt/rocm")
    return os.path.join(rocm, "bin", "hipcc")


def common_flags():
    return [
        f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
        "-I", os.path.join(ROOT, "include"), "-I", CSRC,
        # keep the compiler from emitting packed fp32 arithmetic
        "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
        "-Wno-unused-command-line-argument",
    ]


def _run(cmd):
    p = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    # hipcc's host pass does not know the packed-fp32 feature; drop that warning only
    lines = [l for l in p.stdout.splitlines() if "packed-fp32-ops" not in l and l.strip()]
    if p.returncode != 0:
        raise RuntimeError("build failed: " + " ".join(cmd) + "\n" + "\n".join(lines))
    return lines


def build(verbose: bool = False) -> str:
    """Compile every HIP source and link the shared library; returns its path."""
    os.makedirs(BUILD, exist_ok=True)
    os.makedirs(LIBDIR, exist_ok=True)
    objs, cmds = [], []
    for src in SOURCES:
        obj = os.path.join(BUILD, src.replace(".hip", ".o"))
        objs.append(obj)
        cmds.append([hipcc(), *common_flags(), *EXTRA.get(src, []), "-c", os.path.join(CSRC, src), "-o", obj])
    peaks_tmp = PEAKS + ".tmp"
    cmds.append([hipcc(), *[f for f in common_flags() if f != "-fPIC"], os.path.join(CSRC, PEAKS_SRC), "-o", peaks_tmp])
    with ThreadPoolExecutor(max_workers=min(len(cmds), 8)) as ex:
        for lines in ex.map(_run, cmds):
            if verbose and lines:
                print("\n".join(lines))
    tmp = LIB + ".tmp"
    _run([hipcc(), f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp])
    os.replace(tmp, LIB)
    os.replace(peaks_tmp, PEAKS)
    if verbose:
        print("built", LIB)
    return LIB


if __name__ == "__main__":
    build(verbose=True)
