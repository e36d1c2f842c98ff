"""torch-tensor front-end of the C ABI.

torch supplies device memory and the current HIP stream; every step of the
layer runs in libeqlinear's kernels.  Outputs and the workspace are allocated
here (plumbing) unless the caller passes them in.

Tensor layouts: x [..., Cin, T] (leading dims flattened to N rows),
w [T, Cout, Cin], bias [Cout]; see include/eqlinear.h.
"""
from __future__ import annotations

import torch

from . import _lib

_DT = {torch.float32: _lib.EQL_F32, torch.float16: _lib.EQL_F16}


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype not in _DT:
        raise TypeError("eqlinear supports float32 and float16, got %s" % t.dtype)
    return _DT[t.dtype]


def _ptr(t):
    return None if t is None else (t.data_ptr() or None)


def _stream(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _check_dev(*ts):
    for t in ts:
        if t is not None and not t.is_cuda:
            raise ValueError("eqlinear tensors must live on the GPU")


def weight_spectrum(w: torch.Tensor, out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Opaque weight-spectrum buffer (uint8 tensor) for w [T, Cout, Cin]."""
    _check_dev(w)
    T, Cout, Cin = w.shape
    dt = _dtype_code(w)
    nbytes = _lib.eqlinear_weight_spectrum_bytes(T, Cin, Cout, dt)
    if out is None:
        out = torch.empty(nbytes, dtype=torch.uint8, device=w.device)
    assert out.numel() >= nbytes
    w = w.contiguous()
    _lib.check(_lib.eqlinear_weight_spectrum(_ptr(w), _ptr(out), T, Cin, Cout, dt, _stream(stream)),
               "eqlinear_weight_spectrum")
    return out


def forward(x: torch.Tensor, wspec: torch.Tensor, bias: torch.Tensor | None, T: int, Cin: int,
            Cout: int, out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    _check_dev(x, wspec, bias)
    lead = x.shape[:-2]
    assert tuple(x.shape[-2:]) == (Cin, T), (x.shape, Cin, T)
    x = x.contiguous()
    N = x.numel() // (Cin * T)
    if out is None:
        out = torch.empty(*lead, Cout, T, dtype=x.dtype, device=x.device)
    _lib.check(_lib.eqlinear_forward(_ptr(x), _ptr(wspec), _ptr(bias), _ptr(out), N, T, Cin, Cout,
                                     _dtype_code(x), _stream(stream)), "eqlinear_forward")
    return out


def backward_input(dy: torch.Tensor, wspec: torch.Tensor, T: int, Cin: int, Cout: int,
                   out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    _check_dev(dy, wspec)
    lead = dy.shape[:-2]
    assert tuple(dy.shape[-2:]) == (Cout, T), (dy.shape, Cout, T)
    dy = dy.contiguous()
    N = dy.numel() // (Cout * T)
    if out is None:
        out = torch.empty(*lead, Cin, T, dtype=dy.dtype, device=dy.device)
    _lib.check(_lib.eqlinear_backward_input(_ptr(dy), _ptr(wspec), _ptr(out), N, T, Cin, Cout,
                                            _dtype_code(dy), _stream(stream)),
               "eqlinear_backward_input")
    return out


def workspace_bytes(N: int, T: int, Cin: int, Cout: int, dtype: torch.dtype) -> int:
    return _lib.eqlinear_backward_weight_workspace_bytes(N, T, Cin, Cout, _DT[dtype])


def backward_weight(x: torch.Tensor, dy: torch.Tensor, T: int, Cin: int, Cout: int,
                    with_bias: bool = True, dw: torch.Tensor | None = None,
                    db: torch.Tensor | None = None, workspace: torch.Tensor | None = None,
                    stream=None):
    """(dw [T, Cout, Cin], db [Cout] or None)."""
    _check_dev(x, dy)
    x = x.contiguous()
    dy = dy.contiguous()
    N = x.numel() // (Cin * T)
    assert dy.numel() == N * Cout * T
    dt = _dtype_code(x)
    if dw is None:
        dw = torch.empty(T, Cout, Cin, dtype=x.dtype, device=x.device)
    if with_bias and db is None:
        db = torch.empty(Cout, dtype=x.dtype, device=x.device)
    if not with_bias:
        db = None
    need = _lib.eqlinear_backward_weight_workspace_bytes(N, T, Cin, Cout, dt)
    if workspace is None and need > 0:
        workspace = torch.empty(need, dtype=torch.uint8, device=x.device)
    wsb = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _lib.check(_lib.eqlinear_backward_weight(_ptr(x), _ptr(dy), _ptr(dw), _ptr(db), _ptr(workspace),
                                             wsb, N, T, Cin, Cout, dt, _stream(stream)),
               "eqlinear_backward_weight")
    return dw, db


class EQLinearFunction(torch.autograd.Function):
    """Autograd wrapper: forward through the spectrum, gradients w.r.t. x, w and b."""

    @staticmethod
    def forward(ctx, x, w, b):
        T, Cout, Cin = w.shape
        wspec = weight_spectrum(w)
        ctx.save_for_backward(x, w)
        ctx.wspec = wspec
        ctx.has_bias = b is not None
        return forward(x, wspec, b, T, Cin, Cout)

    @staticmethod
    def backward(ctx, gy):
        x, w = ctx.saved_tensors
        T, Cout, Cin = w.shape
        gy = gy.contiguous()
        gx = gw = gb = None
        if ctx.needs_input_grad[0]:
            gx = backward_input(gy, ctx.wspec, T, Cin, Cout)
        if ctx.needs_input_grad[1] or (ctx.has_bias and ctx.needs_input_grad[2]):
            gw, gb = backward_weight(x, gy, T, Cin, Cout, with_bias=ctx.has_bias)
        return gx, gw, gb


class EQLinear(torch.nn.Module):
    """Equivariant linear layer over C_T: x [..., Cin, T] -> y [..., Cout, T]."""

    def __init__(self, T: int, Cin: int, Cout: int, bias: bool = True, device=None, dtype=None):
        super().__init__()
        self.T, self.Cin, self.Cout = T, Cin, Cout
        kw = {"device": device, "dtype": dtype}
        self.weight = torch.nn.Parameter(torch.randn(T, Cout, Cin, **kw) / (T * Cin) ** 0.5)
        self.bias = torch.nn.Parameter(torch.zeros(Cout, **kw)) if bias else None

    def forward(self, x):
        return EQLinearFunction.apply(x, self.weight, self.bias)
