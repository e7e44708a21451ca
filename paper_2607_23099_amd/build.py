"""In-tree build of the HIP libraries for gfx950.

``build_all()`` compiles
  * ``libdamoe.so``        - the fused-MoE path behind the C-ABI in ``include/damoe.h``
  * ``synth/libdamoe_synth.so`` - the seeded synthetic-input generator
Both are built with hipcc for gfx950 only.
"""
from __future__ import annotations

import glob
import os
import shutil
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
INCLUDE = os.path.join(ROOT, "include")
LIB_DAMOE = os.path.join(PKG, "libdamoe.so")
LIB_SYNTH = os.path.join(PKG, "synth", "libdamoe_synth.so")

ARCH = "gfx950"
# Packed fp32 instructions are kept out of every HIP object.
HIP_FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC", "-shared",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-result",
]


def _hipcc() -> str:
    h = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(h):
        raise RuntimeError("hipcc not found")
    return h


def _run(cmd, verbose):
    if verbose:
        print(" ".join(cmd), flush=True)
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    # The host pass does not know the packed-fp32 feature name; that warning is noise.
    out = "\n".join(l for l in r.stdout.splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"build failed ({r.returncode}):\n{' '.join(cmd)}\n{out}")
    if verbose and out.strip():
        print(out, flush=True)


def _link(sources, out, extra=(), verbose=False):
    tmp = out + ".tmp"
    _run([_hipcc(), *HIP_FLAGS, f"-I{INCLUDE}", *extra, *sources, "-o", tmp], verbose)
    os.replace(tmp, out)


def build_synth(verbose=False):
    _link([os.path.join(PKG, "synth", "synth_fill.hip")], LIB_SYNTH, verbose=verbose)


def damoe_sources():
    return sorted(glob.glob(os.path.join(PKG, "csrc", "*.hip")) +
                  glob.glob(os.path.join(PKG, "csrc", "*.cpp")))


def build_damoe(verbose=False):
    srcs = damoe_sources()
    if not srcs:
        raise RuntimeError("no sources under csrc/")
    _link(srcs, LIB_DAMOE, extra=[f"-I{os.path.join(PKG, 'csrc')}"], verbose=verbose)


def build_all(verbose=False):
    build_synth(verbose)
    if damoe_sources():
        build_damoe(verbose)


if __name__ == "__main__":
    build_all(verbose="-v" in sys.argv)
