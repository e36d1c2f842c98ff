"""Work accounting for the C_T equivariant linear layer: flops, bytes, rooflines.

Counts follow the paper's step-by-step complexity (Sec. 3.3, Theorem 1, and
Appendix A.1), with one refinement: the self-conjugate bins (k = 0, and k = T/2
for even T) are real, so they cost one real product each instead of four.  With
R = 1 + [T even] real bins and K = floor((T-1)/2) complex bins, one pass
(forward, input gradient or weight gradient) contracts (R + 4K) real products
of shape [N, Cin] x [Cin, Cout].  For p4 (T = 4) this is the paper's 6/16 of
the dense cost (Sec. 3.2.2, Step 2).

MI355X peaks are the vendor's published dense figures.
"""
from __future__ import annotations

PEAK_HBM_GBS = 8000.0          # HBM3E, GB/s
PEAK_MFMA_TFLOPS = {"f16": 2516.6, "bf16": 2516.6, "f32": 157.3}   # dense matrix peaks, TFLOP/s
PEAK_FP32_VALU_TFLOPS = 157.3
ELEM_BYTES = {"f32": 4, "f16": 2, "bf16": 2}


def bins(T: int):
    """(R, K): number of real and of complex non-redundant DFT bins of a length-T real signal."""
    R = 1 + (1 if T % 2 == 0 else 0)
    K = (T - 1) // 2
    return R, K


def real_products(T: int) -> int:
    """Real [N,Cin]x[Cin,Cout] products per pass: R + 4K."""
    R, K = bins(T)
    return R + 4 * K


def pass_flops(N, T, Cin, Cout) -> float:
    """Spectral-GEMM flops of one pass (forward, dX or dW)."""
    return 2.0 * real_products(T) * N * Cin * Cout


def dense_equiv_flops(N, T, Cin, Cout) -> float:
    """Flops of the same pass done as a dense unrolled [N, T*Cin] x [T*Cin, T*Cout] GEMM."""
    return 2.0 * N * T * T * Cin * Cout


def paper_flash_flops(N, T, Cin, Cout) -> float:
    """The paper's Table 1 accounting of the Flash forward: 2 * (spectral products + NDT)."""
    return 2.0 * (real_products(T) * N * Cin * Cout + N * Cout * T * T)


def standard_linear_flops(N, C, D) -> float:
    return 2.0 * N * C * D


def eq_params(T, Cin, Cout, bias=True) -> int:
    return T * Cin * Cout + (Cout if bias else 0)


def standard_params(C, D, bias=True) -> int:
    return C * D + (D if bias else 0)


def pass_bytes(kind: str, N, T, Cin, Cout, dtype: str, bias: bool = False) -> float:
    """Algorithmic HBM bytes of one pass: each operand read once, each result written once."""
    e = ELEM_BYTES[dtype]
    a = N * Cin * T * e          # x or dx
    b = N * Cout * T * e         # y or dy
    wb = T * Cin * Cout * e      # weights (or their spectrum) / dw
    bb = Cout * e if bias else 0
    if kind == "fwd":
        return a + b + wb + bb
    if kind == "dx":
        return a + b + wb
    if kind == "dw":
        return a + b + wb + bb
    if kind == "bwd":            # whole backward in one pass: x, dy, spectrum in; dx, dw, db out
        return 2 * a + b + 2 * wb + bb
    if kind == "wspec":
        return 2 * wb
    raise ValueError(kind)


def roofline_time_s(kind, N, T, Cin, Cout, dtype, bias=False) -> float:
    """max(bytes / HBM peak, flops / MFMA peak) for one pass."""
    t_mem = pass_bytes(kind, N, T, Cin, Cout, dtype, bias) / (PEAK_HBM_GBS * 1e9)
    if kind == "wspec":
        return t_mem
    t_mma = pass_flops(N, T, Cin, Cout) * (2 if kind == "bwd" else 1) / (PEAK_MFMA_TFLOPS[dtype] * 1e12)
    return max(t_mem, t_mma)
