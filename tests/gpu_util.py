"""Helpers shared by the GPU tests: run the HIP path on seeded inputs and compare
with the fp64 oracle on the same dtype-rounded values."""
from __future__ import annotations

import sys

import numpy as np

import synth

# max|gpu - ref| / max|ref|, per output tensor.  bf16 (unit roundoff 2^-8)
# takes the fp16 bar (unit roundoff 2^-11) scaled by the ratio, 8.
TOL = {"f32": 1e-5, "f16": 5e-3, "bf16": 4e-2}


def torch_dtype(dt):
    import torch
    return {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}[dt]


def rel_err(gpu, ref):
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    assert gpu.shape == ref.shape, (gpu.shape, ref.shape)
    scale = np.max(np.abs(ref)) if ref.size else 0.0
    if ref.size == 0:
        return 0.0
    if scale == 0.0:
        return float(np.max(np.abs(gpu)))
    return float(np.max(np.abs(gpu - ref)) / scale)


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def to_dev(a, dt):
    """``a`` rounded to dt on the GPU (bf16: the float32-held bf16 values,
    converted exactly)."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(synth.round_to(a, dt))).to("cuda")
    return t.to(torch.bfloat16) if dt == "bf16" else t


def run_gpu(inp: synth.Inputs, dt: str, want=("y", "dx", "dw")):
    """Run weight spectrum, forward, backward_input, backward_weight on the GPU."""
    import torch
    from paper_2607_21271_amd import ops
    T, Cout, Cin = inp.w.shape
    x, w, dy = to_dev(inp.x, dt), to_dev(inp.w, dt), to_dev(inp.dy, dt)
    b = to_dev(inp.b, dt) if inp.b is not None else None
    wspec = ops.weight_spectrum(w)
    out = {}
    if "y" in want:
        out["y"] = ops.forward(x, wspec, b, T, Cin, Cout)
    if "dx" in want:
        out["dx"] = ops.backward_input(dy, wspec, T, Cin, Cout)
    if "dw" in want:
        out["dw"], out["db"] = ops.backward_weight(x, dy, T, Cin, Cout, with_bias=b is not None)
    torch.cuda.synchronize()
    return {k: (v.float().cpu().numpy() if v is not None else None) for k, v in out.items()}
