"""Rotation-equivariant group convolution on a square grid, on the C_T library.

The rotations by 360/T degrees (T in {1, 2, 4}) act on the image plane and on
the group axis of the features; Sec. 5 of the paper names equivariant
convolutions as the next operators to carry the method to.  Features are
f [B, H, W, Cin, T], the weight psi [k, k, T, Cout, Cin] holds one Cout x Cin
block per window offset and group lag, b [Cout]:

    out[n,o,r] = sum_{(a,b)} sum_s sum_c psi[R^-r (a,b)][(s - r) mod T][o][c] f[n + (a,b), c, s] + b[o]

(zero padding, k odd).  Split into rotation orbits of the window, this is one
C_T layer with k*k*Cin input channels on gathered patches
(``eqlinear_gconv_gather``) with a permuted weight
(``eqlinear_gconv_pack_weight``); the forward pass and the gradients run on
the C_T kernels, and ``eqlinear_gconv_scatter`` / ``eqlinear_gconv_unpack_weight``
take the gradients back.  Where Cin is a multiple of 4 the forward kernel
reads the patches straight from f (``eqlinear_gconv_forward``) and no patch
buffer is formed unless the weight gradient needs one.  This module only
allocates and marshals.
"""
from __future__ import annotations

import weakref

import torch

from . import _lib, ops


def _dims(f, Cin, T):
    if f.dim() != 5 or tuple(f.shape[-2:]) != (Cin, T):
        raise ValueError("features must be [B, H, W, Cin=%d, T=%d], got %s" % (Cin, T, tuple(f.shape)))
    return f.shape[0], f.shape[1], f.shape[2]


def gather(f: torch.Tensor, T: int, k: int, stream=None) -> torch.Tensor:
    """xcol [B*H*W, k*k*Cin, T] from f [B, H, W, Cin, T]."""
    Cin = f.shape[-2]
    B, H, W = _dims(f, Cin, T)
    dt = ops._dtype_code(f)
    f = f.contiguous()
    ops._check_dev(f)
    xcol = torch.empty(B * H * W, k * k * Cin, T, dtype=f.dtype, device=f.device)
    _lib.check(_lib.eqlinear_gconv_gather(ops._ptr(f), ops._ptr(xcol), B, H, W, T, Cin, k, dt,
                                          ops._stream(stream)), "eqlinear_gconv_gather")
    return xcol


def scatter(dxcol: torch.Tensor, B: int, H: int, W: int, T: int, Cin: int, k: int, stream=None) -> torch.Tensor:
    """df [B, H, W, Cin, T] from the gradient of xcol (the gather's adjoint)."""
    ops._check_out("dxcol", dxcol, (B * H * W, k * k * Cin, T), dxcol.dtype)
    dt = ops._dtype_code(dxcol)
    ops._check_dev(dxcol)
    df = torch.empty(B, H, W, Cin, T, dtype=dxcol.dtype, device=dxcol.device)
    _lib.check(_lib.eqlinear_gconv_scatter(ops._ptr(dxcol), ops._ptr(df), B, H, W, T, Cin, k, dt,
                                           ops._stream(stream)), "eqlinear_gconv_scatter")
    return df


def pack_weight(psi: torch.Tensor, stream=None) -> torch.Tensor:
    """w_ct [T, Cout, k*k*Cin] from psi [k, k, T, Cout, Cin]."""
    if psi.dim() != 5 or psi.shape[0] != psi.shape[1]:
        raise ValueError("psi must be [k, k, T, Cout, Cin], got %s" % (tuple(psi.shape),))
    k, _, T, Cout, Cin = psi.shape
    dt = ops._dtype_code(psi)
    psi = psi.contiguous()
    ops._check_dev(psi)
    w = torch.empty(T, Cout, k * k * Cin, dtype=psi.dtype, device=psi.device)
    _lib.check(_lib.eqlinear_gconv_pack_weight(ops._ptr(psi), ops._ptr(w), T, Cin, Cout, k, dt,
                                               ops._stream(stream)), "eqlinear_gconv_pack_weight")
    return w


def pack_weight_adjoint(psi: torch.Tensor, stream=None) -> torch.Tensor:
    """w_adj [T, Cin, k*k*Cout] from psi [k, k, T, Cout, Cin]: the C_T weight of
    the adjoint convolution (``eqlinear_gconv_pack_weight_adjoint``), which
    maps the output gradient [B, H, W, Cout, T] to the input gradient."""
    if psi.dim() != 5 or psi.shape[0] != psi.shape[1]:
        raise ValueError("psi must be [k, k, T, Cout, Cin], got %s" % (tuple(psi.shape),))
    k, _, T, Cout, Cin = psi.shape
    dt = ops._dtype_code(psi)
    psi = psi.contiguous()
    ops._check_dev(psi)
    w = torch.empty(T, Cin, k * k * Cout, dtype=psi.dtype, device=psi.device)
    _lib.check(_lib.eqlinear_gconv_pack_weight_adjoint(ops._ptr(psi), ops._ptr(w), T, Cin, Cout, k, dt,
                                                       ops._stream(stream)), "eqlinear_gconv_pack_weight_adjoint")
    return w


def unpack_weight_grad(dw_ct: torch.Tensor, k: int, stream=None) -> torch.Tensor:
    """dpsi [k, k, T, Cout, Cin] from the gradient of w_ct [T, Cout, k*k*Cin]."""
    T, Cout, C2 = dw_ct.shape
    if C2 % (k * k):
        raise ValueError("dw_ct channels %d are not a multiple of k*k = %d" % (C2, k * k))
    Cin = C2 // (k * k)
    ops._check_out("dw_ct", dw_ct, (T, Cout, C2), dw_ct.dtype)
    dt = ops._dtype_code(dw_ct)
    ops._check_dev(dw_ct)
    dpsi = torch.empty(k, k, T, Cout, Cin, dtype=dw_ct.dtype, device=dw_ct.device)
    _lib.check(_lib.eqlinear_gconv_unpack_weight(ops._ptr(dw_ct), ops._ptr(dpsi), T, Cin, Cout, k, dt,
                                                 ops._stream(stream)), "eqlinear_gconv_unpack_weight")
    return dpsi


def forward_implicit(f: torch.Tensor, wspec: torch.Tensor, bias, T: int, Cout: int, k: int, stream=None):
    """y [B, H, W, Cout, T] with the forward kernel reading the patches straight
    from f [B, H, W, Cin, T] (``eqlinear_gconv_forward``; needs Cin % 4 == 0);
    bit for bit the result of gather followed by ``ops.forward``."""
    Cin = f.shape[-2]
    B, H, W = _dims(f, Cin, T)
    ops._check_same_dtype(f, bias=bias)
    f = f.contiguous()
    dt = ops._dtype_code(f)
    ops._check_wspec(wspec, T, k * k * Cin, Cout, f.dtype)
    ops._check_dev(f, wspec, *([bias] if bias is not None else []))
    if bias is not None:
        ops._check_out("bias", bias, (Cout,), f.dtype)
    y = torch.empty(B, H, W, Cout, T, dtype=f.dtype, device=f.device)
    _lib.check(_lib.eqlinear_gconv_forward(ops._ptr(f), ops._ptr(wspec), ops._ptr(bias) if bias is not None else None,
                                           ops._ptr(y), B, H, W, T, Cin, Cout, k, dt, ops._stream(stream)),
               "eqlinear_gconv_forward")
    return y


def implicit_ok(Cin: int) -> bool:
    """Whether ``forward_implicit`` takes this layer (its lanes read four
    gathered channels of one block, so Cin must be a multiple of 4)."""
    return Cin % 4 == 0


# C_T weights and spectrum per psi (forward and adjoint), reused while psi's
# storage and version counter (bumped by in-place updates) and the stream are
# unchanged.
_CACHE: dict = {}
_CACHE_ADJ: dict = {}


def _cached(cache, psi: torch.Tensor, pack):
    stream = torch.cuda.current_stream(psi.device).cuda_stream
    key = (psi.data_ptr(), psi._version, tuple(psi.shape), psi.dtype, stream)
    ent = cache.get(id(psi))
    if ent is not None and ent[0]() is psi and ent[1] == key:
        return ent[2]
    w_ct = pack(psi)
    val = (w_ct, ops.weight_spectrum(w_ct))
    pid = id(psi)
    cache[pid] = (weakref.ref(psi, lambda _r, pid=pid: cache.pop(pid, None)), key, val)
    return val


def cached_ct_weight(psi: torch.Tensor):
    return _cached(_CACHE, psi, pack_weight)


def cached_adjoint_weight(psi: torch.Tensor):
    return _cached(_CACHE_ADJ, psi, pack_weight_adjoint)


class GroupConv2dFunction(torch.autograd.Function):
    """Autograd: f [B, H, W, Cin, T], psi [k, k, T, Cout, Cin], b [Cout] or None.

    Input gradient: where Cout is a multiple of 4, the adjoint convolution of
    the output gradient (``pack_weight_adjoint``) through the implicit-gather
    forward, so neither the patch gradient nor its scatter is formed; else
    the C_T input gradient of the patches and ``scatter``.  Weight gradient:
    the C_T weight gradient of the gathered patches."""

    @staticmethod
    def forward(ctx, f, psi, b):
        ops._check_same_dtype(f, psi=psi, b=b)
        k, _, T, Cout, Cin = psi.shape
        B, H, W = _dims(f, Cin, T)
        _, wspec = cached_ct_weight(psi)
        f = f.contiguous()
        want_w = ctx.needs_input_grad[1] or (b is not None and ctx.needs_input_grad[2])
        if implicit_ok(Cin) and not want_w:
            # patches read straight from f (no patch buffer); the weight
            # gradient, which needs them, takes the explicit gather below
            y = forward_implicit(f, wspec, b, T, Cout, k)
            ctx.save_for_backward(f, psi)
            ctx.xcol_saved = False
        else:
            xcol = gather(f, T, k)
            y = ops.forward(xcol, wspec, b, T, k * k * Cin, Cout).view(B, H, W, Cout, T)
            ctx.save_for_backward(xcol, psi)
            ctx.xcol_saved = True
        ctx.wspec, ctx.dims, ctx.has_bias = wspec, (B, H, W, T, Cin, Cout, k), b is not None
        return y

    @staticmethod
    def backward(ctx, gy):
        saved, psi = ctx.saved_tensors
        B, H, W, T, Cin, Cout, k = ctx.dims
        want_w = ctx.needs_input_grad[1] or (ctx.has_bias and ctx.needs_input_grad[2])
        xcol = saved if ctx.xcol_saved else (gather(saved, T, k) if want_w else None)
        C2 = k * k * Cin
        gy = gy.contiguous()
        gy2 = gy.view(B * H * W, Cout, T)
        gf = gpsi = gb = None
        dx2 = dw2 = None
        if ctx.needs_input_grad[0] and implicit_ok(Cout):
            _, wspec_adj = cached_adjoint_weight(psi)
            gf = forward_implicit(gy, wspec_adj, None, T, Cin, k)
            if want_w:
                dw2, gb = ops.backward_weight(xcol, gy2, T, C2, Cout, with_bias=ctx.has_bias)
        elif ctx.needs_input_grad[0] and want_w:
            dx2, dw2, gb = ops.backward(xcol, gy2, ctx.wspec, T, C2, Cout, with_bias=ctx.has_bias)
        elif ctx.needs_input_grad[0]:
            dx2 = ops.backward_input(gy2, ctx.wspec, T, C2, Cout)
        elif want_w:
            dw2, gb = ops.backward_weight(xcol, gy2, T, C2, Cout, with_bias=ctx.has_bias)
        if dx2 is not None:
            gf = scatter(dx2, B, H, W, T, Cin, k)
        if dw2 is not None:
            gpsi = unpack_weight_grad(dw2, k)
        return gf, gpsi, gb


class GroupConv2d(torch.nn.Module):
    """Rotation-equivariant k x k group convolution: [B, H, W, Cin, T] -> [B, H, W, Cout, T]."""

    def __init__(self, T: int, Cin: int, Cout: int, k: int = 3, bias: bool = True, device=None, dtype=None):
        super().__init__()
        self.T, self.Cin, self.Cout, self.k = T, Cin, Cout, k
        kw = {"device": device, "dtype": dtype}
        self.weight = torch.nn.Parameter(torch.randn(k, k, T, Cout, Cin, **kw) / (k * k * T * Cin) ** 0.5)
        self.bias = torch.nn.Parameter(torch.zeros(Cout, **kw)) if bias else None

    def forward(self, f):
        return GroupConv2dFunction.apply(f, self.weight, self.bias)
