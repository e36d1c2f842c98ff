"""Equivariant linear layer over the dihedral group D_T on the C_T library.

D_T holds the T rotations and T reflections of a regular T-gon; Sec. 5 of the
paper names reflection groups as the next groups to cover.  Elements
(t, m) = r^t s^m are stored at m*T + t, so features are x [..., Cin, 2T]
(2T group positions per channel), the weight W [2T, Cout, Cin] holds one
Cout x Cin block per group element and b [Cout] one bias per channel.  The
layer shares weights by the group law, as the C_T layer does (Sec. 3.1,
Eq. 1-2):

    y[n,o,g] = sum_h sum_c W[h^-1 g][o][c] x[n,c,h] + b[o].

Read as [N, 2Cin, T], x is the input of a C_T layer with 2Cin -> 2Cout
channels whose weight is gathered from W (``eqlinear_dihedral_expand``, see
include/eqlinear.h), so the forward pass and the gradients run on the C_T
kernels (weight spectrum, forward, whole backward) and the gradients with
respect to W and b are folded back by ``eqlinear_dihedral_fold``.  Every step
runs in libeqlinear's kernels; this module only allocates and marshals.
"""
from __future__ import annotations

import weakref

import torch

from . import _lib, ops


def _check(t, name, shape, dtype):
    if tuple(t.shape) != tuple(shape):
        raise ValueError("%s has shape %s, expected %s" % (name, tuple(t.shape), tuple(shape)))
    if t.dtype != dtype:
        raise TypeError("%s has dtype %s, expected %s" % (name, t.dtype, dtype))
    if not t.is_contiguous():
        raise ValueError("%s must be contiguous" % name)


def expand(w: torch.Tensor, b: torch.Tensor | None = None, stream=None):
    """(w_ct [T, 2Cout, 2Cin], b_ct [2Cout] or None): the C_T layer's weights."""
    if w.dim() != 3 or w.shape[0] % 2:
        raise ValueError("w must be [2T, Cout, Cin], got shape %s" % (tuple(w.shape),))
    G, Cout, Cin = w.shape
    T = G // 2
    dt = ops._dtype_code(w)
    w = w.contiguous()
    if b is not None:
        _check(b.contiguous(), "b", (Cout,), w.dtype)
        b = b.contiguous()
    ops._check_dev(w, b)
    w_ct = torch.empty(T, 2 * Cout, 2 * Cin, dtype=w.dtype, device=w.device)
    b_ct = torch.empty(2 * Cout, dtype=w.dtype, device=w.device) if b is not None else None
    _lib.check(_lib.eqlinear_dihedral_expand(ops._ptr(w), ops._ptr(b), ops._ptr(w_ct), ops._ptr(b_ct), T,
                                             Cin, Cout, dt, ops._stream(stream)),
               "eqlinear_dihedral_expand")
    return w_ct, b_ct


def fold(dw_ct: torch.Tensor, db_ct: torch.Tensor | None = None, stream=None):
    """(dW [2T, Cout, Cin], db [Cout] or None) from the C_T layer's gradients."""
    if dw_ct.dim() != 3 or dw_ct.shape[1] % 2 or dw_ct.shape[2] % 2:
        raise ValueError("dw_ct must be [T, 2Cout, 2Cin], got shape %s" % (tuple(dw_ct.shape),))
    T, O2, C2 = dw_ct.shape
    Cout, Cin = O2 // 2, C2 // 2
    dt = ops._dtype_code(dw_ct)
    _check(dw_ct, "dw_ct", (T, O2, C2), dw_ct.dtype)
    if db_ct is not None:
        _check(db_ct, "db_ct", (O2,), dw_ct.dtype)
    ops._check_dev(dw_ct, db_ct)
    dW = torch.empty(2 * T, Cout, Cin, dtype=dw_ct.dtype, device=dw_ct.device)
    db = torch.empty(Cout, dtype=dw_ct.dtype, device=dw_ct.device) if db_ct is not None else None
    _lib.check(_lib.eqlinear_dihedral_fold(ops._ptr(dw_ct), ops._ptr(db_ct), ops._ptr(dW), ops._ptr(db), T,
                                           Cin, Cout, dt, ops._stream(stream)),
               "eqlinear_dihedral_fold")
    return dW, db


# C_T weights and spectrum per (W, b), reused while neither tensor's storage or
# version counter (bumped by in-place updates) nor the stream changes.
_CACHE: dict = {}


def cached_ct_weights(w: torch.Tensor, b: torch.Tensor | None):
    stream = torch.cuda.current_stream(w.device).cuda_stream
    key = (w.data_ptr(), w._version, tuple(w.shape), w.dtype, stream,
           None if b is None else (b.data_ptr(), b._version))
    ent = _CACHE.get(id(w))
    if ent is not None and ent[0]() is w and ent[1] == key:
        return ent[2]
    w_ct, b_ct = expand(w, b)
    val = (w_ct, b_ct, ops.weight_spectrum(w_ct))
    wid = id(w)
    _CACHE[wid] = (weakref.ref(w, lambda _r, wid=wid: _CACHE.pop(wid, None)), key, val)
    return val


class DihedralEQLinearFunction(torch.autograd.Function):
    """Autograd over D_T: x [..., Cin, 2T], w [2T, Cout, Cin], b [Cout] or None."""

    @staticmethod
    def forward(ctx, x, w, b):
        ops._check_same_dtype(x, w=w, b=b)
        G, Cout, Cin = w.shape
        T = G // 2
        if G % 2 or tuple(x.shape[-2:]) != (Cin, G):
            raise ValueError("x must be [..., Cin=%d, 2T=%d], got %s" % (Cin, G, tuple(x.shape)))
        x = x.contiguous()
        lead = x.shape[:-2]
        N = x.numel() // (Cin * G)
        _, b_ct, wspec = cached_ct_weights(w, b)
        y = ops.forward(x.view(N, 2 * Cin, T), wspec, b_ct, T, 2 * Cin, 2 * Cout)
        ctx.save_for_backward(x)
        ctx.wspec, ctx.T, ctx.Cin, ctx.Cout, ctx.has_bias = wspec, T, Cin, Cout, b is not None
        return y.view(*lead, Cout, G)

    @staticmethod
    def backward(ctx, gy):
        (x,) = ctx.saved_tensors
        T, Cin, Cout = ctx.T, ctx.Cin, ctx.Cout
        N = x.numel() // (Cin * 2 * T)
        x2 = x.view(N, 2 * Cin, T)
        gy2 = gy.contiguous().view(N, 2 * Cout, T)
        gx = gw = gb = None
        want_w = ctx.needs_input_grad[1] or (ctx.has_bias and ctx.needs_input_grad[2])
        dx2 = dw2 = db2 = None
        if ctx.needs_input_grad[0] and want_w:
            dx2, dw2, db2 = ops.backward(x2, gy2, ctx.wspec, T, 2 * Cin, 2 * Cout, with_bias=ctx.has_bias)
        elif ctx.needs_input_grad[0]:
            dx2 = ops.backward_input(gy2, ctx.wspec, T, 2 * Cin, 2 * Cout)
        elif want_w:
            dw2, db2 = ops.backward_weight(x2, gy2, T, 2 * Cin, 2 * Cout, with_bias=ctx.has_bias)
        if dx2 is not None:
            gx = dx2.view(x.shape)
        if dw2 is not None:
            gw, gb = fold(dw2, db2)
        return gx, gw, gb


class DihedralEQLinear(torch.nn.Module):
    """Equivariant linear layer over D_T: x [..., Cin, 2T] -> y [..., Cout, 2T]."""

    def __init__(self, T: int, Cin: int, Cout: int, bias: bool = True, device=None, dtype=None):
        super().__init__()
        self.T, self.Cin, self.Cout = T, Cin, Cout
        kw = {"device": device, "dtype": dtype}
        self.weight = torch.nn.Parameter(torch.randn(2 * T, Cout, Cin, **kw) / (2 * T * Cin) ** 0.5)
        self.bias = torch.nn.Parameter(torch.zeros(Cout, **kw)) if bias else None

    def forward(self, x):
        return DihedralEQLinearFunction.apply(x, self.weight, self.bias)
