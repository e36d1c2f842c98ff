"""Build libeqlinear.so (gfx950) in-tree with hipcc.

Each translation unit is compiled in its own hipcc process (in parallel), then
linked into ``paper_2607_21271_amd/libeqlinear.so``.  The kernel instantiations
are one object per (group order T, dtype): ``eql_inst.hip`` compiled 48 times.  Always rebuilds.  The
device assembly is kept (-save-temps) and scanned by isa_check before the
library is installed; a finding fails the build.
Usage: ``python -m paper_2607_21271_amd.build`` or ``build()``.
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import shutil
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
OUT = os.path.join(HERE, "libeqlinear.so")
BUILD_DIR = os.path.join(HERE, "_build")

HOST_SOURCES = ["eql_api.cpp", "eql_dispatch.cpp"]
MAX_T = 16
# (source, object stem, extra defines)
UNITS = [("eql_big.hip", "eql_big", [])] + [(s, os.path.splitext(s)[0], []) for s in HOST_SOURCES] + [
    ("eql_inst.hip", "inst_%s_t%02d" % (name, t), ["-DEQK_T=%d" % t, "-DEQK_DT=%d" % dt])
    for t in range(MAX_T, 0, -1) for dt, name in ((1, "f16"), (0, "f32"), (2, "bf16"))]

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
# Packed-fp32 instructions are switched off for all device code.
# MFMA accumulators may live in arch VGPRs (gfx950 has a unified register
# file); with this selection the kernels of two waves per SIMD allocate
# without scratch.  The large-tile unit (one wave per SIMD, T * 64
# accumulators per lane) keeps them in the accumulation registers instead.
LINK_FLAGS = ["--offload-arch=" + ARCH, "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
VGPR_FORM = ["-mllvm", "-amdgpu-mfma-vgpr-form=1"]
DEVICE_FLAGS = LINK_FLAGS + VGPR_FORM
ACC_REG_UNITS = {"eql_big"}
COMMON_FLAGS = ["-O3", "-std=c++20", "-fPIC", "-Wall", "-Wno-unused-function",
                "-I" + os.path.join(os.path.dirname(HERE), "include")]


def _compile(unit) -> str:
    src, stem, defs = unit
    wd = os.path.join(BUILD_DIR, stem)   # -save-temps names its files after the source
    os.makedirs(wd, exist_ok=True)
    obj = os.path.join(wd, stem + ".o")
    lang = ["-x", "hip"] if src.endswith(".cpp") else []
    dev = LINK_FLAGS if stem in ACC_REG_UNITS else DEVICE_FLAGS
    cmd = [HIPCC, *dev, *COMMON_FLAGS, *defs, "-save-temps", *lang, "-c",
           os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True, cwd=wd)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed for %s:\n%s\n%s" % (src, " ".join(cmd), r.stderr[-20000:]))
    return obj


def build(verbose: bool = True) -> str:
    shutil.rmtree(BUILD_DIR, ignore_errors=True)
    os.makedirs(BUILD_DIR, exist_ok=True)
    jobs = min(len(UNITS), int(os.environ.get("MAX_JOBS", os.cpu_count() or 4)))
    with cf.ThreadPoolExecutor(max_workers=max(1, jobs)) as ex:
        objs = list(ex.map(_compile, UNITS))
    from . import isa_check
    isa_check.check_build(BUILD_DIR)
    tmp = OUT + ".tmp%d" % os.getpid()
    cmd = [HIPCC, *DEVICE_FLAGS, "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n%s\n%s" % (" ".join(cmd), r.stderr[-20000:]))
    os.replace(tmp, OUT)
    if verbose:
        print("built", OUT)
    return OUT


def clean():
    shutil.rmtree(BUILD_DIR, ignore_errors=True)


if __name__ == "__main__":
    build()
    sys.exit(0)
