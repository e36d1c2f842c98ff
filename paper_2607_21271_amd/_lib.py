"""ctypes binding of libeqlinear.so: the C ABI of include/eqlinear.h, same names.

Argument marshalling only.  Every function takes device addresses as Python
ints (or None for NULL) and returns the library's status code; ``check``
turns a non-zero status into an ``EqlError``.  Loading fails loudly when the
library has not been built: there is no fallback implementation.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libeqlinear.so")

EQL_F32 = 0
EQL_F16 = 1
EQL_BF16 = 2

EQL_OK = 0
EQL_ERR_INVALID_ARG = 1
EQL_ERR_UNSUPPORTED = 2
EQL_ERR_ALIGNMENT = 3
EQL_ERR_WORKSPACE = 4
EQL_ERR_NO_DEVICE = 5
EQL_ERR_LAUNCH = 6
EQL_ERR_SCRATCH = 7

# Bytes of the static device scratch of eqlinear_backward_weight_noalloc
# (EQLINEAR_STATIC_SCRATCH_BYTES in include/eqlinear.h).
STATIC_SCRATCH_BYTES = 64 << 20

# Every function the header declares, with (restype, argtypes).
_vp, _i, _i64, _sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_size_t
SIGNATURES = {
    "eqlinear_abi_version": (_i, []),
    "eqlinear_status_string": (ctypes.c_char_p, [_i]),
    "eqlinear_weight_spectrum_bytes": (_sz, [_i, _i, _i, _i]),
    "eqlinear_weight_spectrum": (_i, [_vp, _vp, _i, _i, _i, _i, _vp]),
    "eqlinear_forward": (_i, [_vp, _vp, _vp, _vp, _i64, _i, _i, _i, _i, _vp]),
    "eqlinear_backward_input": (_i, [_vp, _vp, _vp, _i64, _i, _i, _i, _i, _vp]),
    "eqlinear_backward_weight_workspace_bytes": (_sz, [_i64, _i, _i, _i, _i]),
    "eqlinear_backward_weight": (_i, [_vp, _vp, _vp, _vp, _vp, _sz, _i64, _i, _i, _i, _i, _vp]),
    "eqlinear_backward_weight_noalloc": (_i, [_vp, _vp, _vp, _vp, _i64, _i, _i, _i, _i, _vp]),
    "eqlinear_backward_workspace_bytes": (_sz, [_i64, _i, _i, _i, _i]),
    "eqlinear_backward_is_fused": (_i, [_i64, _i, _i, _i, _i]),
    "eqlinear_backward": (_i, [_vp, _vp, _vp, _vp, _vp, _vp, _vp, _sz, _i64, _i, _i, _i, _i, _vp]),
    "eqlinear_dihedral_expand": (_i, [_vp, _vp, _vp, _vp, _i, _i, _i, _i, _vp]),
    "eqlinear_dihedral_fold": (_i, [_vp, _vp, _vp, _vp, _i, _i, _i, _i, _vp]),
    "eqlinear_gconv_gather": (_i, [_vp, _vp, _i64, _i, _i, _i, _i, _i, _i, _vp]),
    "eqlinear_gconv_scatter": (_i, [_vp, _vp, _i64, _i, _i, _i, _i, _i, _i, _vp]),
    "eqlinear_gconv_pack_weight": (_i, [_vp, _vp, _i, _i, _i, _i, _i, _vp]),
    "eqlinear_gconv_pack_weight_adjoint": (_i, [_vp, _vp, _i, _i, _i, _i, _i, _vp]),
    "eqlinear_gconv_unpack_weight": (_i, [_vp, _vp, _i, _i, _i, _i, _i, _vp]),
    "eqlinear_gconv_forward": (_i, [_vp, _vp, _vp, _vp, _i64, _i, _i, _i, _i, _i, _i, _i, _vp]),
}


class EqlError(RuntimeError):
    def __init__(self, status: int, where: str = ""):
        self.status = status
        super().__init__("%s: status %d (%s)" % (where or "eqlinear", status, status_string(status)))


_lib = None


def lib(path: str | None = None):
    """Load libeqlinear.so (cached).  Raises if it is missing."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise RuntimeError("libeqlinear.so is not built (%s); run __graft_entry__.build() or "
                           "python -m paper_2607_21271_amd.build" % p)
    handle = ctypes.CDLL(p)
    for name, (res, args) in SIGNATURES.items():
        f = getattr(handle, name)
        f.restype = res
        f.argtypes = args
    if path is None:
        _lib = handle
    return handle


def status_string(status: int) -> str:
    return lib().eqlinear_status_string(status).decode()


def check(status: int, where: str = "") -> None:
    if status != EQL_OK:
        raise EqlError(status, where)


def eqlinear_abi_version() -> int:
    return lib().eqlinear_abi_version()


def eqlinear_status_string(status: int) -> str:
    return status_string(status)


def eqlinear_weight_spectrum_bytes(T, Cin, Cout, dtype) -> int:
    return lib().eqlinear_weight_spectrum_bytes(T, Cin, Cout, dtype)


def eqlinear_weight_spectrum(w, wspec, T, Cin, Cout, dtype, stream) -> int:
    return lib().eqlinear_weight_spectrum(w, wspec, T, Cin, Cout, dtype, stream)


def eqlinear_forward(x, wspec, bias, y, N, T, Cin, Cout, dtype, stream) -> int:
    return lib().eqlinear_forward(x, wspec, bias, y, N, T, Cin, Cout, dtype, stream)


def eqlinear_backward_input(dy, wspec, dx, N, T, Cin, Cout, dtype, stream) -> int:
    return lib().eqlinear_backward_input(dy, wspec, dx, N, T, Cin, Cout, dtype, stream)


def eqlinear_backward_weight_workspace_bytes(N, T, Cin, Cout, dtype) -> int:
    return lib().eqlinear_backward_weight_workspace_bytes(N, T, Cin, Cout, dtype)


def eqlinear_backward_weight(x, dy, dw, dbias, workspace, workspace_bytes, N, T, Cin, Cout, dtype,
                             stream) -> int:
    return lib().eqlinear_backward_weight(x, dy, dw, dbias, workspace, workspace_bytes, N, T, Cin,
                                          Cout, dtype, stream)


def eqlinear_backward_weight_noalloc(x, dy, dw, dbias, N, T, Cin, Cout, dtype, stream) -> int:
    return lib().eqlinear_backward_weight_noalloc(x, dy, dw, dbias, N, T, Cin, Cout, dtype, stream)


def eqlinear_backward_workspace_bytes(N, T, Cin, Cout, dtype) -> int:
    return lib().eqlinear_backward_workspace_bytes(N, T, Cin, Cout, dtype)


def eqlinear_backward_is_fused(N, T, Cin, Cout, dtype) -> int:
    return lib().eqlinear_backward_is_fused(N, T, Cin, Cout, dtype)


def eqlinear_backward(x, dy, wspec, dx, dw, dbias, workspace, workspace_bytes, N, T, Cin, Cout, dtype,
                      stream) -> int:
    return lib().eqlinear_backward(x, dy, wspec, dx, dw, dbias, workspace, workspace_bytes, N, T, Cin,
                                   Cout, dtype, stream)


def eqlinear_dihedral_expand(w, bias, w_ct, bias_ct, T, Cin, Cout, dtype, stream) -> int:
    return lib().eqlinear_dihedral_expand(w, bias, w_ct, bias_ct, T, Cin, Cout, dtype, stream)


def eqlinear_dihedral_fold(dw_ct, dbias_ct, dw, dbias, T, Cin, Cout, dtype, stream) -> int:
    return lib().eqlinear_dihedral_fold(dw_ct, dbias_ct, dw, dbias, T, Cin, Cout, dtype, stream)


def eqlinear_gconv_gather(f, xcol, B, H, W, T, Cin, k, dtype, stream) -> int:
    return lib().eqlinear_gconv_gather(f, xcol, B, H, W, T, Cin, k, dtype, stream)


def eqlinear_gconv_scatter(dxcol, df, B, H, W, T, Cin, k, dtype, stream) -> int:
    return lib().eqlinear_gconv_scatter(dxcol, df, B, H, W, T, Cin, k, dtype, stream)


def eqlinear_gconv_pack_weight(psi, w_ct, T, Cin, Cout, k, dtype, stream) -> int:
    return lib().eqlinear_gconv_pack_weight(psi, w_ct, T, Cin, Cout, k, dtype, stream)


def eqlinear_gconv_pack_weight_adjoint(psi, w_adj, T, Cin, Cout, k, dtype, stream) -> int:
    return lib().eqlinear_gconv_pack_weight_adjoint(psi, w_adj, T, Cin, Cout, k, dtype, stream)


def eqlinear_gconv_unpack_weight(dw_ct, dpsi, T, Cin, Cout, k, dtype, stream) -> int:
    return lib().eqlinear_gconv_unpack_weight(dw_ct, dpsi, T, Cin, Cout, k, dtype, stream)


def eqlinear_gconv_forward(f, wspec, bias, y, B, H, W, T, Cin, Cout, k, dtype, stream) -> int:
    return lib().eqlinear_gconv_forward(f, wspec, bias, y, B, H, W, T, Cin, Cout, k, dtype, stream)
