"""fp64 CPU oracle for the C_T equivariant linear layer (arXiv 2607.21271).

TEST INFRASTRUCTURE ONLY.  Imported by the tests, by ``__graft_entry__.smoke()``
and by the ``cpu_baseline`` leg of ``bench.py`` -- nowhere else.  The GPU
library never loads it and shares no code with it.

The arithmetic lives in ``eqref.c`` (the defining circular-convolution sums of
Sec. 3.1, Eq. 1-2, with the convolution lag direction; see that file's header).
This module only compiles it with gcc and marshals numpy arrays through ctypes.
Every input is converted to a contiguous float64 array first, so callers pass
the dtype-rounded values they also hand to the GPU.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "eqref.c")
_LIB_PATH = os.path.join(_HERE, "libeqref.so")
CFLAGS = ["-O2", "-fno-fast-math", "-ffp-contract=off", "-fopenmp", "-fPIC", "-shared",
          "-std=c11", "-Wall", "-Wextra"]

_lib = None


def build(src: str = _SRC, out: str = _LIB_PATH, extra_flags=()) -> str:
    """Compile ``src`` into a shared library at ``out`` (always recompiles)."""
    tmp = out + ".tmp%d" % os.getpid()
    cmd = ["gcc", *CFLAGS, *extra_flags, src, "-o", tmp]
    subprocess.run(cmd, check=True)
    os.replace(tmp, out)
    return out


_D = ctypes.POINTER(ctypes.c_double)
_I32 = ctypes.POINTER(ctypes.c_int32)
_i64 = ctypes.c_int64
_int = ctypes.c_int


def load(path: str | None = None):
    """Load the compiled oracle (building it if absent) and declare signatures."""
    global _lib
    if path is None and _lib is not None:
        return _lib
    p = path or _LIB_PATH
    if path is None and (not os.path.exists(p) or os.path.getmtime(p) < os.path.getmtime(_SRC)):
        build()
    lib = ctypes.CDLL(p)
    lib.eqref_forward.argtypes = [_D, _D, _D, _D, _i64, _int, _int, _int]
    lib.eqref_backward_input.argtypes = [_D, _D, _D, _i64, _int, _int, _int]
    lib.eqref_backward_weight.argtypes = [_D, _D, _D, _D, _i64, _int, _int, _int]
    lib.eqref_backward_weight_entries.argtypes = [_D, _D, _I32, _I32, _I32, _i64, _D,
                                                  _i64, _int, _int, _int]
    for f in (lib.eqref_forward, lib.eqref_backward_input, lib.eqref_backward_weight,
              lib.eqref_backward_weight_entries):
        f.restype = None
    if path is None:
        _lib = lib
    return lib


def _f64(a):
    return np.ascontiguousarray(np.asarray(a, dtype=np.float64))


def _ptr(a):
    return a.ctypes.data_as(_D) if a is not None else None


class Oracle:
    """Thin numpy front-end over one compiled copy of ``eqref.c``."""

    def __init__(self, lib=None):
        self.lib = lib if lib is not None else load()

    def forward(self, x, w, b=None):
        """y[N,Cout,T] from x[N,Cin,T], w[T,Cout,Cin], b[Cout] or None."""
        x, w = _f64(x), _f64(w)
        b = _f64(b) if b is not None else None
        N, Cin, T = x.shape
        Tw, Cout, Cin_w = w.shape
        assert Tw == T and Cin_w == Cin
        y = np.empty((N, Cout, T), np.float64)
        self.lib.eqref_forward(_ptr(x), _ptr(w), _ptr(b), _ptr(y), N, T, Cin, Cout)
        return y

    def backward_input(self, dy, w):
        """dx[N,Cin,T] from dy[N,Cout,T] and w[T,Cout,Cin]."""
        dy, w = _f64(dy), _f64(w)
        N, Cout, T = dy.shape
        Tw, Cout_w, Cin = w.shape
        assert Tw == T and Cout_w == Cout
        dx = np.empty((N, Cin, T), np.float64)
        self.lib.eqref_backward_input(_ptr(dy), _ptr(w), _ptr(dx), N, T, Cin, Cout)
        return dx

    def backward_weight(self, x, dy, with_bias=True):
        """(dw[T,Cout,Cin], db[Cout] or None) from x[N,Cin,T] and dy[N,Cout,T]."""
        x, dy = _f64(x), _f64(dy)
        N, Cin, T = x.shape
        N2, Cout, T2 = dy.shape
        assert N2 == N and T2 == T
        dw = np.empty((T, Cout, Cin), np.float64)
        db = np.empty((Cout,), np.float64) if with_bias else None
        self.lib.eqref_backward_weight(_ptr(x), _ptr(dy), _ptr(dw), _ptr(db), N, T, Cin, Cout)
        return dw, db

    def backward_weight_entries(self, x, dy, j, o, c):
        """dw[j[e], o[e], c[e]] for each sampled entry e."""
        x, dy = _f64(x), _f64(dy)
        N, Cin, T = x.shape
        Cout = dy.shape[1]
        j = np.ascontiguousarray(j, np.int32)
        o = np.ascontiguousarray(o, np.int32)
        c = np.ascontiguousarray(c, np.int32)
        out = np.empty(j.shape, np.float64)
        self.lib.eqref_backward_weight_entries(
            _ptr(x), _ptr(dy), j.ctypes.data_as(_I32), o.ctypes.data_as(_I32),
            c.ctypes.data_as(_I32), j.size, _ptr(out), N, T, Cin, Cout)
        return out


_default = None


def oracle() -> Oracle:
    global _default
    if _default is None:
        _default = Oracle()
    return _default


def forward(x, w, b=None):
    return oracle().forward(x, w, b)


def backward_input(dy, w):
    return oracle().backward_input(dy, w)


def backward_weight(x, dy, with_bias=True):
    return oracle().backward_weight(x, dy, with_bias)


def backward_weight_entries(x, dy, j, o, c):
    return oracle().backward_weight_entries(x, dy, j, o, c)


# ---------------------------------------------------------------------------
# Dihedral group D_T (eqref_dihedral.c): the same weight-sharing layer over the
# rotations and reflections of a regular T-gon.  Group index g = m*T + t
# (t the rotation, m the reflection bit); x [N, Cin, 2T], W [2T, Cout, Cin].

_DSRC = os.path.join(_HERE, "eqref_dihedral.c")
_DLIB_PATH = os.path.join(_HERE, "libeqref_dihedral.so")
_dlib = None


def load_dihedral(path: str | None = None):
    """Load the compiled dihedral oracle (building it if absent)."""
    global _dlib
    if path is None and _dlib is not None:
        return _dlib
    p = path or _DLIB_PATH
    if path is None and (not os.path.exists(p) or os.path.getmtime(p) < os.path.getmtime(_DSRC)):
        build(_DSRC, _DLIB_PATH)
    lib = ctypes.CDLL(p)
    lib.eqref_dihedral_forward.argtypes = [_D, _D, _D, _D, _i64, _int, _int, _int]
    lib.eqref_dihedral_backward_input.argtypes = [_D, _D, _D, _i64, _int, _int, _int]
    lib.eqref_dihedral_backward_weight.argtypes = [_D, _D, _D, _D, _i64, _int, _int, _int]
    for f in (lib.eqref_dihedral_forward, lib.eqref_dihedral_backward_input,
              lib.eqref_dihedral_backward_weight):
        f.restype = None
    lib.eqref_dihedral_mul.argtypes = [_int, _int, _int]
    lib.eqref_dihedral_mul.restype = _int
    lib.eqref_dihedral_inv.argtypes = [_int, _int]
    lib.eqref_dihedral_inv.restype = _int
    if path is None:
        _dlib = lib
    return lib


class DihedralOracle:
    """numpy front-end over the compiled D_T oracle."""

    def __init__(self, lib=None):
        self.lib = lib if lib is not None else load_dihedral()

    def mul(self, a, b, T):
        return self.lib.eqref_dihedral_mul(a, b, T)

    def inv(self, a, T):
        return self.lib.eqref_dihedral_inv(a, T)

    def forward(self, x, W, b=None):
        """y[N,Cout,2T] from x[N,Cin,2T], W[2T,Cout,Cin], b[Cout] or None."""
        x, W = _f64(x), _f64(W)
        b = _f64(b) if b is not None else None
        N, Cin, G = x.shape
        Gw, Cout, Cin_w = W.shape
        assert Gw == G and Cin_w == Cin and G % 2 == 0
        y = np.empty((N, Cout, G), np.float64)
        self.lib.eqref_dihedral_forward(_ptr(x), _ptr(W), _ptr(b), _ptr(y), N, G // 2, Cin, Cout)
        return y

    def backward_input(self, dy, W):
        """dx[N,Cin,2T] from dy[N,Cout,2T] and W[2T,Cout,Cin]."""
        dy, W = _f64(dy), _f64(W)
        N, Cout, G = dy.shape
        Gw, Cout_w, Cin = W.shape
        assert Gw == G and Cout_w == Cout
        dx = np.empty((N, Cin, G), np.float64)
        self.lib.eqref_dihedral_backward_input(_ptr(dy), _ptr(W), _ptr(dx), N, G // 2, Cin, Cout)
        return dx

    def backward_weight(self, x, dy, with_bias=True):
        """(dW[2T,Cout,Cin], db[Cout] or None) from x[N,Cin,2T] and dy[N,Cout,2T]."""
        x, dy = _f64(x), _f64(dy)
        N, Cin, G = x.shape
        N2, Cout, G2 = dy.shape
        assert N2 == N and G2 == G
        dW = np.empty((G, Cout, Cin), np.float64)
        db = np.empty((Cout,), np.float64) if with_bias else None
        self.lib.eqref_dihedral_backward_weight(_ptr(x), _ptr(dy), _ptr(dW), _ptr(db), N, G // 2,
                                                Cin, Cout)
        return dW, db


_ddefault = None


def dihedral_oracle() -> DihedralOracle:
    global _ddefault
    if _ddefault is None:
        _ddefault = DihedralOracle()
    return _ddefault


# ---------------------------------------------------------------------------
# Rotation-equivariant group convolution on a square grid (eqref_gconv.c):
# f [B, H, W, Cin, T], psi [k, k, T, Cout, Cin], out [B, H, W, Cout, T],
# T in {1, 2, 4}, k odd.

_GSRC = os.path.join(_HERE, "eqref_gconv.c")
_GLIB_PATH = os.path.join(_HERE, "libeqref_gconv.so")
_glib = None


def load_gconv(path: str | None = None):
    """Load the compiled group-convolution oracle (building it if absent)."""
    global _glib
    if path is None and _glib is not None:
        return _glib
    p = path or _GLIB_PATH
    if path is None and (not os.path.exists(p) or os.path.getmtime(p) < os.path.getmtime(_GSRC)):
        build(_GSRC, _GLIB_PATH)
    lib = ctypes.CDLL(p)
    dims = [_int] * 7
    lib.eqref_gconv_forward.argtypes = [_D, _D, _D, _D] + dims
    lib.eqref_gconv_backward_input.argtypes = [_D, _D, _D] + dims
    lib.eqref_gconv_backward_weight.argtypes = [_D, _D, _D, _D] + dims
    for f in (lib.eqref_gconv_forward, lib.eqref_gconv_backward_input, lib.eqref_gconv_backward_weight):
        f.restype = None
    if path is None:
        _glib = lib
    return lib


class GconvOracle:
    """numpy front-end over the compiled group-convolution oracle."""

    def __init__(self, lib=None):
        self.lib = lib if lib is not None else load_gconv()

    def forward(self, f, psi, bias=None):
        f, psi = _f64(f), _f64(psi)
        bias = _f64(bias) if bias is not None else None
        B, H, W, Cin, T = f.shape
        k, k2, T2, Cout, Cin2 = psi.shape
        assert k == k2 and k % 2 == 1 and T2 == T and Cin2 == Cin
        out = np.empty((B, H, W, Cout, T), np.float64)
        self.lib.eqref_gconv_forward(_ptr(f), _ptr(psi), _ptr(bias), _ptr(out), B, H, W, T, Cin, Cout, k)
        return out

    def backward_input(self, dout, psi):
        dout, psi = _f64(dout), _f64(psi)
        B, H, W, Cout, T = dout.shape
        k, _, _, Cout2, Cin = psi.shape
        assert Cout2 == Cout
        df = np.empty((B, H, W, Cin, T), np.float64)
        self.lib.eqref_gconv_backward_input(_ptr(dout), _ptr(psi), _ptr(df), B, H, W, T, Cin, Cout, k)
        return df

    def backward_weight(self, f, dout, k, with_bias=True):
        f, dout = _f64(f), _f64(dout)
        B, H, W, Cin, T = f.shape
        Cout = dout.shape[3]
        dpsi = np.empty((k, k, T, Cout, Cin), np.float64)
        db = np.empty((Cout,), np.float64) if with_bias else None
        self.lib.eqref_gconv_backward_weight(_ptr(f), _ptr(dout), _ptr(dpsi), _ptr(db), B, H, W, T, Cin,
                                             Cout, k)
        return dpsi, db


_gdefault = None


def gconv_oracle() -> GconvOracle:
    global _gdefault
    if _gdefault is None:
        _gdefault = GconvOracle()
    return _gdefault
