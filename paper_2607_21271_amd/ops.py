"""torch-tensor front-end of the C ABI.

torch supplies device memory and the current HIP stream; every step of the
layer runs in libeqlinear's kernels.  Outputs and the workspace are allocated
here (plumbing) unless the caller passes them in.

Tensor layouts: x [..., Cin, T] (leading dims flattened to N rows),
w [T, Cout, Cin], bias [Cout]; see include/eqlinear.h.

The C ABI receives raw device addresses only, so every check that needs the
tensors themselves happens here, before any launch: all tensors of a call live
on one GPU and share one dtype (float32, float16 or bfloat16), outputs that the caller
passes in are contiguous with exactly the expected shape, and a weight
spectrum is a contiguous uint8 buffer of exactly
``eqlinear_weight_spectrum_bytes`` bytes for the call's (T, Cin, Cout, dtype)
(an fp32 spectrum is twice the size of a 16-bit one, so a spectrum of the
wrong width is refused; fp16 and bf16 spectra have the same size, so the
caller keeps a spectrum with the dtype it was computed for, as
``EQLinearFunction`` does).
"""
from __future__ import annotations

import weakref

import torch

from . import _lib

_DT = {torch.float32: _lib.EQL_F32, torch.float16: _lib.EQL_F16, torch.bfloat16: _lib.EQL_BF16}


def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype not in _DT:
        raise TypeError("eqlinear supports float32, float16 and bfloat16, got %s" % t.dtype)
    return _DT[t.dtype]


def _ptr(t):
    return None if t is None else (t.data_ptr() or None)


def _stream(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _check_dev(*ts):
    dev = None
    for t in ts:
        if t is None:
            continue
        if not t.is_cuda:
            raise ValueError("eqlinear tensors must live on the GPU")
        if dev is None:
            dev = t.device
        elif t.device != dev:
            raise ValueError("eqlinear tensors of one call must be on one device (%s vs %s)"
                             % (dev, t.device))


def _check_same_dtype(ref: torch.Tensor, **named):
    for name, t in named.items():
        if t is not None and t.dtype != ref.dtype:
            raise TypeError("%s has dtype %s, expected %s (one dtype per call)"
                            % (name, t.dtype, ref.dtype))


def _check_out(name: str, t, shape, dtype):
    if t is None:
        return
    if tuple(t.shape) != tuple(shape):
        raise ValueError("%s has shape %s, expected %s" % (name, tuple(t.shape), tuple(shape)))
    if t.dtype != dtype:
        raise TypeError("%s has dtype %s, expected %s" % (name, t.dtype, dtype))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)


def spectrum_bytes(T: int, Cin: int, Cout: int, dtype: torch.dtype) -> int:
    return _lib.eqlinear_weight_spectrum_bytes(T, Cin, Cout, _DT[dtype])


def _check_wspec(wspec: torch.Tensor, T, Cin, Cout, dtype):
    need = spectrum_bytes(T, Cin, Cout, dtype)
    if wspec.dtype != torch.uint8 or wspec.dim() != 1 or not wspec.is_contiguous():
        raise TypeError("a weight spectrum is a contiguous 1-d uint8 buffer")
    if wspec.numel() != need:
        raise ValueError("weight spectrum has %d bytes; (T=%d, Cin=%d, Cout=%d, %s) needs exactly %d"
                         % (wspec.numel(), T, Cin, Cout, dtype, need))


def weight_spectrum(w: torch.Tensor, out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Opaque weight-spectrum buffer (uint8 tensor) for w [T, Cout, Cin]."""
    if w.dim() != 3:
        raise ValueError("w must be [T, Cout, Cin], got shape %s" % (tuple(w.shape),))
    T, Cout, Cin = w.shape
    dt = _dtype_code(w)
    if out is not None:
        _check_wspec(out, T, Cin, Cout, w.dtype)
    _check_dev(w, out)
    nbytes = _lib.eqlinear_weight_spectrum_bytes(T, Cin, Cout, dt)
    if out is None:
        out = torch.empty(nbytes, dtype=torch.uint8, device=w.device)
    w = w.contiguous()
    _lib.check(_lib.eqlinear_weight_spectrum(_ptr(w), _ptr(out), T, Cin, Cout, dt, _stream(stream)),
               "eqlinear_weight_spectrum")
    return out


def forward(x: torch.Tensor, wspec: torch.Tensor, bias: torch.Tensor | None, T: int, Cin: int,
            Cout: int, out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    dt = _dtype_code(x)
    _check_same_dtype(x, bias=bias)
    if tuple(x.shape[-2:]) != (Cin, T):
        raise ValueError("x must be [..., Cin=%d, T=%d], got %s" % (Cin, T, tuple(x.shape)))
    if bias is not None and tuple(bias.shape) != (Cout,):
        raise ValueError("bias must be [Cout=%d], got %s" % (Cout, tuple(bias.shape)))
    _check_wspec(wspec, T, Cin, Cout, x.dtype)
    lead = x.shape[:-2]
    _check_out("out", out, tuple(lead) + (Cout, T), x.dtype)
    _check_dev(x, wspec, bias, out)
    x = x.contiguous()
    bias = None if bias is None else bias.contiguous()
    N = x.numel() // (Cin * T)
    if out is None:
        out = torch.empty(*lead, Cout, T, dtype=x.dtype, device=x.device)
    _lib.check(_lib.eqlinear_forward(_ptr(x), _ptr(wspec), _ptr(bias), _ptr(out), N, T, Cin, Cout,
                                     dt, _stream(stream)), "eqlinear_forward")
    return out


def backward_input(dy: torch.Tensor, wspec: torch.Tensor, T: int, Cin: int, Cout: int,
                   out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    dt = _dtype_code(dy)
    if tuple(dy.shape[-2:]) != (Cout, T):
        raise ValueError("dy must be [..., Cout=%d, T=%d], got %s" % (Cout, T, tuple(dy.shape)))
    _check_wspec(wspec, T, Cin, Cout, dy.dtype)
    lead = dy.shape[:-2]
    _check_out("out", out, tuple(lead) + (Cin, T), dy.dtype)
    _check_dev(dy, wspec, out)
    dy = dy.contiguous()
    N = dy.numel() // (Cout * T)
    if out is None:
        out = torch.empty(*lead, Cin, T, dtype=dy.dtype, device=dy.device)
    _lib.check(_lib.eqlinear_backward_input(_ptr(dy), _ptr(wspec), _ptr(out), N, T, Cin, Cout,
                                            dt, _stream(stream)), "eqlinear_backward_input")
    return out


def workspace_bytes(N: int, T: int, Cin: int, Cout: int, dtype: torch.dtype) -> int:
    return _lib.eqlinear_backward_weight_workspace_bytes(N, T, Cin, Cout, _DT[dtype])


def backward_weight(x: torch.Tensor, dy: torch.Tensor, T: int, Cin: int, Cout: int,
                    with_bias: bool = True, dw: torch.Tensor | None = None,
                    db: torch.Tensor | None = None, workspace: torch.Tensor | None = None,
                    stream=None):
    """(dw [T, Cout, Cin], db [Cout] or None)."""
    dt = _dtype_code(x)
    _check_same_dtype(x, dy=dy)
    if tuple(x.shape[-2:]) != (Cin, T) or tuple(dy.shape[-2:]) != (Cout, T):
        raise ValueError("x must be [..., %d, %d] and dy [..., %d, %d], got %s and %s"
                         % (Cin, T, Cout, T, tuple(x.shape), tuple(dy.shape)))
    N = x.numel() // (Cin * T)
    if dy.numel() != N * Cout * T:
        raise ValueError("x and dy must have the same number of rows")
    if not with_bias:
        db = None
    _check_out("dw", dw, (T, Cout, Cin), x.dtype)
    _check_out("db", db, (Cout,), x.dtype)
    need = _lib.eqlinear_backward_weight_workspace_bytes(N, T, Cin, Cout, dt)
    if workspace is not None:
        if workspace.dim() != 1 or not workspace.is_contiguous():
            raise ValueError("workspace must be a contiguous 1-d buffer")
        if workspace.numel() * workspace.element_size() < need:
            raise ValueError("workspace has %d bytes, needs %d"
                             % (workspace.numel() * workspace.element_size(), need))
    _check_dev(x, dy, dw, db, workspace)
    x = x.contiguous()
    dy = dy.contiguous()
    if dw is None:
        dw = torch.empty(T, Cout, Cin, dtype=x.dtype, device=x.device)
    if with_bias and db is None:
        db = torch.empty(Cout, dtype=x.dtype, device=x.device)
    if workspace is None and need > 0:
        workspace = torch.empty(need, dtype=torch.uint8, device=x.device)
    wsb = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _lib.check(_lib.eqlinear_backward_weight(_ptr(x), _ptr(dy), _ptr(dw), _ptr(db), _ptr(workspace),
                                             wsb, N, T, Cin, Cout, dt, _stream(stream)),
               "eqlinear_backward_weight")
    return dw, db


def backward_weight_noalloc(x: torch.Tensor, dy: torch.Tensor, T: int, Cin: int, Cout: int,
                            dw: torch.Tensor, db: torch.Tensor | None = None, stream=None):
    """dw [T, Cout, Cin] (and db [Cout] when given) through the allocation-free
    entry point: outputs are caller-provided and nothing is allocated, on the
    host or the device (the split partials use the library's static device
    scratch; calls that overlap on one GPU must not be issued)."""
    dt = _dtype_code(x)
    _check_same_dtype(x, dy=dy)
    if tuple(x.shape[-2:]) != (Cin, T) or tuple(dy.shape[-2:]) != (Cout, T):
        raise ValueError("x must be [..., %d, %d] and dy [..., %d, %d], got %s and %s"
                         % (Cin, T, Cout, T, tuple(x.shape), tuple(dy.shape)))
    if not (x.is_contiguous() and dy.is_contiguous()):
        raise ValueError("x and dy must be contiguous (no copies are made)")
    N = x.numel() // (Cin * T)
    if dy.numel() != N * Cout * T:
        raise ValueError("x and dy must have the same number of rows")
    _check_out("dw", dw, (T, Cout, Cin), x.dtype)
    _check_out("db", db, (Cout,), x.dtype)
    _check_dev(x, dy, dw, db)
    _lib.check(_lib.eqlinear_backward_weight_noalloc(_ptr(x), _ptr(dy), _ptr(dw), _ptr(db), N, T, Cin,
                                                     Cout, dt, _stream(stream)),
               "eqlinear_backward_weight_noalloc")
    return dw, db


def backward_workspace_bytes(N: int, T: int, Cin: int, Cout: int, dtype: torch.dtype) -> int:
    return _lib.eqlinear_backward_workspace_bytes(N, T, Cin, Cout, _DT[dtype])


def backward_is_fused(N: int, T: int, Cin: int, Cout: int, dtype: torch.dtype) -> bool:
    """True if ``backward`` runs this problem as one fused pass over x and dy."""
    return bool(_lib.eqlinear_backward_is_fused(N, T, Cin, Cout, _DT[dtype]))


def backward(x: torch.Tensor, dy: torch.Tensor, wspec: torch.Tensor, T: int, Cin: int, Cout: int,
             with_bias: bool = True, dx: torch.Tensor | None = None, dw: torch.Tensor | None = None,
             db: torch.Tensor | None = None, workspace: torch.Tensor | None = None, stream=None):
    """(dx [..., Cin, T], dw [T, Cout, Cin], db [Cout] or None) in one call of
    eqlinear_backward (one fused pass where the library plans one)."""
    dt = _dtype_code(x)
    _check_same_dtype(x, dy=dy)
    if tuple(x.shape[-2:]) != (Cin, T) or tuple(dy.shape[-2:]) != (Cout, T):
        raise ValueError("x must be [..., %d, %d] and dy [..., %d, %d], got %s and %s"
                         % (Cin, T, Cout, T, tuple(x.shape), tuple(dy.shape)))
    N = x.numel() // (Cin * T)
    if dy.numel() != N * Cout * T:
        raise ValueError("x and dy must have the same number of rows")
    _check_wspec(wspec, T, Cin, Cout, x.dtype)
    if not with_bias:
        db = None
    lead = x.shape[:-2]
    _check_out("dx", dx, tuple(lead) + (Cin, T), x.dtype)
    _check_out("dw", dw, (T, Cout, Cin), x.dtype)
    _check_out("db", db, (Cout,), x.dtype)
    need = _lib.eqlinear_backward_workspace_bytes(N, T, Cin, Cout, dt)
    if workspace is not None:
        if workspace.dim() != 1 or not workspace.is_contiguous():
            raise ValueError("workspace must be a contiguous 1-d buffer")
        if workspace.numel() * workspace.element_size() < need:
            raise ValueError("workspace has %d bytes, needs %d"
                             % (workspace.numel() * workspace.element_size(), need))
    _check_dev(x, dy, wspec, dx, dw, db, workspace)
    x = x.contiguous()
    dy = dy.contiguous()
    if dx is None:
        dx = torch.empty(*lead, Cin, T, dtype=x.dtype, device=x.device)
    if dw is None:
        dw = torch.empty(T, Cout, Cin, dtype=x.dtype, device=x.device)
    if with_bias and db is None:
        db = torch.empty(Cout, dtype=x.dtype, device=x.device)
    if workspace is None and need > 0:
        workspace = torch.empty(need, dtype=torch.uint8, device=x.device)
    wsb = 0 if workspace is None else workspace.numel() * workspace.element_size()
    _lib.check(_lib.eqlinear_backward(_ptr(x), _ptr(dy), _ptr(wspec), _ptr(dx), _ptr(dw), _ptr(db),
                                      _ptr(workspace), wsb, N, T, Cin, Cout, dt, _stream(stream)),
               "eqlinear_backward")
    return dx, dw, db


# Weight spectra of the autograd path, per weight tensor: reused while the
# weight's storage, version counter (bumped by every in-place update, e.g. an
# optimizer step) and the current stream are unchanged.  Keyed by id() with a
# weak reference to the tensor (tensors do not compare as dictionary keys); an
# entry leaves the cache when its tensor is freed.
_SPEC_CACHE: dict = {}


def cached_weight_spectrum(w: torch.Tensor) -> torch.Tensor:
    stream = torch.cuda.current_stream(w.device).cuda_stream
    key = (w.data_ptr(), w._version, tuple(w.shape), w.dtype, stream)
    ent = _SPEC_CACHE.get(id(w))
    if ent is not None and ent[0]() is w and ent[1] == key:
        return ent[2]
    spec = weight_spectrum(w)
    wid = id(w)
    ref = weakref.ref(w, lambda _r, wid=wid: _SPEC_CACHE.pop(wid, None))
    _SPEC_CACHE[wid] = (ref, key, spec)
    return spec


class EQLinearFunction(torch.autograd.Function):
    """Autograd wrapper: forward through the spectrum, gradients w.r.t. x, w and b."""

    @staticmethod
    def forward(ctx, x, w, b):
        _check_same_dtype(x, w=w, b=b)
        T, Cout, Cin = w.shape
        wspec = cached_weight_spectrum(w)
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
        want_w = ctx.needs_input_grad[1] or (ctx.has_bias and ctx.needs_input_grad[2])
        if ctx.needs_input_grad[0] and want_w:
            gx, gw, gb = backward(x, gy, ctx.wspec, T, Cin, Cout, with_bias=ctx.has_bias)
        elif ctx.needs_input_grad[0]:
            gx = backward_input(gy, ctx.wspec, T, Cin, Cout)
        elif want_w:
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
