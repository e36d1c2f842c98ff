"""Post-build scan of the gfx950 assembly of libeqlinear.so.

The fp16 activation words are unpacked by one inline-asm statement per word
(``f16x2_to_f32`` in csrc/eql_common.h): a convert of the low half into an
early-clobber output, then a convert of the high half.  In some kernels this
toolchain's register allocator once gave that output the input's register (the
word then reads as already converted), and before the asm form, the same fault
showed as a word being overwritten between its two half-conversions.  Both
miscompiles give wrong numbers without any error, so the build scans the
device assembly for them and refuses to produce a library that has either.

Checks, per kernel:
  clobbered_unpack   the unpack asm's first convert writes its own input register
  converted_source   an f16->f32 convert reads a register whose last write in
                     the same basic block was an fp32 result (a raw word is
                     never such a value)
  mfma_dst_overlap   an MFMA whose result spans more than four registers has a
                     destination that partially overlaps its accumulator
                     input (srcC).  The gfx950 assembler refuses exactly this
                     form ("source 2 operand must not partially overlap with
                     dst") and accepts partial overlap for four-register
                     results, which the compiler emits for the 16x16 MFMAs
                     of these kernels; the check keeps a build from carrying
                     the refused form in code that bypassed the assembler's
                     operand validation.
  fused_scratch      a single-pass backward kernel (eql_bwd_fused_kernel) uses
                     scratch memory: only variants that fit the registers are
                     built, and a spilling one would run far slower than the
                     two-kernel path the host would otherwise have chosen.
"""
from __future__ import annotations

import glob
import os
import re
import subprocess

_FUNC = re.compile(r"^(_Z\S+):")
_BLOCK_END = re.compile(r"^\.LBB|^\s*s_cbranch|^\s*s_branch|^; %bb")
_CVT = re.compile(r"^\s*v_cvt_f32_f16\S*\s+v(\d+),\s*v(\d+)\b")
_F32_DEF = re.compile(r"^\s*(v_cvt_f32_f16\S*|v_add_f32\S*|v_sub_f32\S*|v_subrev_f32\S*|v_mul_f32\S*"
                      r"|v_fma_f32\S*|v_fmac_f32\S*|v_fmamk_f32\S*|v_fmaak_f32\S*)\s+v(\d+),")
_DEF_RANGE = re.compile(r"^\s*(v_\S+|buffer_load\S*|global_load\S*|ds_read\S*)\s+v\[(\d+):(\d+)\]")
_DEF_ONE = re.compile(r"^\s*(v_\S+|buffer_load\S*|global_load\S*|ds_read\S*)\s+v(\d+)\b")
_UNPACK_FIRST = re.compile(r"^\s*v_cvt_f32_f16_e32 v(\d+), v(\d+)\s*$")
_SCRATCH = re.compile(r"^; ScratchSize: (\d+)")
_MFMA = re.compile(r"^\s*v_mfma\S*\s+([va])\[(\d+):(\d+)\],\s*[^,]+,\s*[^,]+,\s*([va])\[(\d+):(\d+)\]")


def scan_lines(lines):
    """Return a list of (kernel, check, instruction) problems found in assembly lines."""
    problems = []
    kernel = None
    last = {}          # vgpr -> "f32" | "other", within the current basic block
    in_asm = False
    asm_first = False
    for line in lines:
        m = _FUNC.match(line)
        if m:
            kernel, last, in_asm = m.group(1), {}, False
            continue
        if "ASMSTART" in line:
            in_asm, asm_first = True, True
            continue
        if "ASMEND" in line:
            in_asm = False
            continue
        sc = _SCRATCH.match(line)
        if sc and kernel and "eql_bwd_fused_kernel" in kernel and int(sc.group(1)) > 0:
            problems.append((kernel, "fused_scratch", line.strip()))
            continue
        if _BLOCK_END.match(line):
            last = {}
            continue
        if in_asm and asm_first:
            asm_first = False
            u = _UNPACK_FIRST.match(line)
            if u and u.group(1) == u.group(2):
                problems.append((kernel, "clobbered_unpack", line.strip()))
        mf = _MFMA.match(line)
        if mf:
            d0, d1, c0, c1 = (int(mf.group(i)) for i in (2, 3, 5, 6))
            if (mf.group(1) == mf.group(4) and d1 - d0 + 1 > 4 and (d0, d1) != (c0, c1)
                    and d0 <= c1 and c0 <= d1):
                problems.append((kernel, "mfma_dst_overlap", line.strip()))
        c = _CVT.match(line)
        if c and last.get(int(c.group(2))) == "f32":
            problems.append((kernel, "converted_source", line.strip()))
        f = _F32_DEF.match(line)
        if f:
            last[int(f.group(2))] = "f32"
            continue
        r = _DEF_RANGE.match(line)
        if r:
            for k in range(int(r.group(2)), int(r.group(3)) + 1):
                last[k] = "other"
            continue
        d = _DEF_ONE.match(line)
        if d and not line.strip().startswith("v_cmp"):
            last[int(d.group(2))] = "other"
    return problems


def scan_file(path):
    with open(path) as f:
        return scan_lines(f)


def device_asm_files(build_dir):
    return sorted(glob.glob(os.path.join(build_dir, "**", "*-hip-amdgcn-amd-amdhsa-*.s"), recursive=True))


def demangle(names):
    try:
        out = subprocess.run(["c++filt"], input="\n".join(names), capture_output=True, text=True).stdout
        return out.split("\n")[: len(names)]
    except OSError:
        return list(names)


def check_build(build_dir):
    """Scan every device assembly file of a build; raise RuntimeError on a problem."""
    files = device_asm_files(build_dir)
    if not files:
        raise RuntimeError("no device assembly found in %s (the build keeps it with -save-temps)" % build_dir)
    problems = []
    for path in files:
        problems += [(os.path.basename(path),) + p for p in scan_file(path)]
    if problems:
        names = demangle([p[1] for p in problems])
        msg = "\n".join("  %s: %s: %s: %s" % (p[0], n, p[2], p[3]) for p, n in zip(problems[:20], names))
        raise RuntimeError("device code failed the post-build check (%d findings):\n%s"
                           % (len(problems), msg))
    return files
