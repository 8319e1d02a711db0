"""Build ``liblutgemm.so`` for gfx950 with hipcc (in-tree, no JIT cache).

Every HIP source is compiled to an object under ``_build/`` and linked into
``paper_2408_06003_amd/liblutgemm.so``.  Flags: -O3, no FP contraction (the
INT8 activation quantizer and the FP32 output rounding must follow the
definition exactly), correctly rounded FP32 division, and packed-FP32
instructions disabled; code object version 5, which every ROCm 7 runtime
(including the one bundled with PyTorch) loads.

``build(timeline=True)`` (``python build.py --timeline``) builds an instrumented
variant, ``liblutgemm_timeline.so``, compiled with ``-DLUTGEMM_TIMELINE``: lane 0 of
every wavefront of the single-token kernels records real-time-clock stamps at its
phase boundaries into a buffer given with ``lutgemm_timeline_set`` (see
``timeline.py``).  The product library is never built with it.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
CSRC = os.path.join(HERE, "csrc")
BUILD = os.path.join(ROOT, "_build")
LIB = os.path.join(HERE, "liblutgemm.so")
TIMELINE_LIB = os.path.join(HERE, "liblutgemm_timeline.so")
SOURCES = ["api.cpp", "pack.hip", "precompute.hip", "lut_gemv.hip", "lut_mpgemm.hip", "lut_fused.hip", "lut_mtok.hip", "lut_tri.hip", "dequant_mfma.hip", "calib.hip", "noalloc.hip"]
ARCH = "gfx950"

COMMON = [
    "-O3", "-std=c++17", "-fPIC", f"--offload-arch={ARCH}", "-mcode-object-version=5",
    "-ffp-contract=off", "-fhip-fp32-correctly-rounded-divide-sqrt",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-command-line-argument",
    f"-I{os.path.join(ROOT, 'include')}",
]


def _compile(src: str, timeline: bool = False) -> str:
    bdir = os.path.join(BUILD, "timeline") if timeline else BUILD
    os.makedirs(bdir, exist_ok=True)
    obj = os.path.join(bdir, os.path.splitext(src)[0] + ".o")
    lang = ["-x", "hip"]
    extra = ["-DLUTGEMM_TIMELINE"] if timeline else []
    cmd = ["hipcc", *lang, *COMMON, *extra, "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"hipcc failed for {src}:\n{r.stdout}\n{r.stderr}")
    return obj


def build(verbose: bool = True, timeline: bool = False) -> str:
    """Compile every source for gfx950 and link the shared library; returns its path."""
    with cf.ThreadPoolExecutor(max_workers=min(len(SOURCES), os.cpu_count() or 4)) as ex:
        objs = list(ex.map(lambda src: _compile(src, timeline), SOURCES))
    lib = TIMELINE_LIB if timeline else LIB
    tmp = lib + ".tmp"
    cmd = ["hipcc", f"--offload-arch={ARCH}", "-mcode-object-version=5", "-shared", "-fPIC", "-o", tmp, *objs]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError(f"link failed:\n{r.stdout}\n{r.stderr}")
    os.replace(tmp, lib)
    if verbose:
        print(f"built {lib}")
    return lib


if __name__ == "__main__":
    build(timeline="--timeline" in sys.argv)
    sys.exit(0)
