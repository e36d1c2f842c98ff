"""The three-product (Gauss) forms of a complex bin's product that the fp32
large-tile kernels take at T = 4, checked on the CPU against plain complex
matrix products (numpy complex128).  Each form splits one complex GEMM of
Eq. 5 into three real GEMMs accumulated apart and combined afterwards:

  forward         Y = X W^T:        A1 = (Xr + Xi) Wr^T, A2 = Xr (Wi - Wr)^T,
                                    A3 = Xi (Wr + Wi)^T;  Re = A1 - A3, Im = A1 + A2
  input gradient  dX = dY conj(W):  A1 = (Dr + Di) Wr,   A2 = Di (Wi - Wr),
                                    A3 = Dr (Wr + Wi);    Re = A1 + A2, Im = A1 - A3
  weight gradient H = conj(X)^T dY: A1 = (Xr - Xi)^T Dr, A2 = Xr^T (Di - Dr),
                                    A3 = Xi^T (Dr + Di);  Re = A1 + A3, Im = A1 + A2

(the combinations the kernels form in registers; the four-product forms are
the plain complex products).  A wrong sign or a swapped operand in any of
them fails here.
"""
import numpy as np
import pytest


def _cplx(rs, *shape):
    return rs.standard_normal(shape) + 1j * rs.standard_normal(shape)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_forward_three_products(seed):
    rs = np.random.RandomState(seed)
    X, W = _cplx(rs, 37, 24), _cplx(rs, 19, 24)
    Xr, Xi, Wr, Wi = X.real, X.imag, W.real, W.imag
    A1 = (Xr + Xi) @ Wr.T
    A2 = Xr @ (Wi - Wr).T
    A3 = Xi @ (Wr + Wi).T
    ref = X @ W.T
    np.testing.assert_allclose(A1 - A3, ref.real, rtol=0, atol=1e-10)
    np.testing.assert_allclose(A1 + A2, ref.imag, rtol=0, atol=1e-10)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_input_gradient_three_products(seed):
    rs = np.random.RandomState(seed)
    D, W = _cplx(rs, 37, 19), _cplx(rs, 19, 24)   # dY [N, Cout], W [Cout, Cin]
    Dr, Di, Wr, Wi = D.real, D.imag, W.real, W.imag
    A1 = (Dr + Di) @ Wr
    A2 = Di @ (Wi - Wr)
    A3 = Dr @ (Wr + Wi)
    ref = D @ np.conj(W)
    np.testing.assert_allclose(A1 + A2, ref.real, rtol=0, atol=1e-10)
    np.testing.assert_allclose(A1 - A3, ref.imag, rtol=0, atol=1e-10)


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_weight_gradient_three_products(seed):
    rs = np.random.RandomState(seed)
    X, D = _cplx(rs, 41, 24), _cplx(rs, 41, 19)   # rows are the contraction
    Xr, Xi, Dr, Di = X.real, X.imag, D.real, D.imag
    A1 = (Xr - Xi).T @ Dr
    A2 = Xr.T @ (Di - Dr)
    A3 = Xi.T @ (Dr + Di)
    ref = np.conj(X).T @ D
    np.testing.assert_allclose(A1 + A3, ref.real, rtol=0, atol=1e-10)
    np.testing.assert_allclose(A1 + A2, ref.imag, rtol=0, atol=1e-10)


def test_three_forms_fail_on_a_planted_sign():
    """The check is sharp: flipping the sign that combines A3 breaks it."""
    rs = np.random.RandomState(5)
    X, W = _cplx(rs, 8, 6), _cplx(rs, 5, 6)
    A1 = (X.real + X.imag) @ W.real.T
    A3 = X.imag @ (W.real + W.imag).T
    assert not np.allclose(A1 + A3, (X @ W.T).real)
