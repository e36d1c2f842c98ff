"""Pins of the dihedral-group oracle (oracle/eqref_dihedral.c) on the CPU.

The layer over D_T is the weight-sharing rule of the C_T layer (Sec. 3.1,
Eq. 1-2) applied with the group law of D_T (Sec. 5 names reflection groups
as the next groups to cover).  The oracle is pinned against facts that do not
come from it:

* its group law is D_T: the presentation <r, s | r^T = s^2 = 1, s r s = r^-1>,
  the storage order g = m*T + t = r^t s^m, associativity and inverses;
* equivariance: translating the input by any element translates the output;
* D_1 is the cyclic group of order 2, so the layer equals the (separately
  pinned) C_T oracle at T = 2;
* D_2 is the Klein four-group Z2 x Z2, so the layer is a 2-d circular
  convolution, computed here with numpy's 2-d FFT;
* inputs on the rotations only with reflection blocks zero reduce to the C_T
  layer;
* the gradients are the adjoints of the forward map (bilinear identities).
A set of planted mistakes in copies of the source is caught by these pins.
"""
import os
import shutil
import tempfile

import numpy as np
import pytest

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(os.path.dirname(HERE), "oracle", "eqref_dihedral.c")


@pytest.fixture(scope="module")
def d():
    return oracle.dihedral_oracle()


def _rand(seed, *shape):
    return np.random.RandomState(seed).standard_normal(shape)


def _power(d, a, k, T):
    e = 0
    for _ in range(k):
        e = d.mul(e, a, T)
    return e


@pytest.mark.parametrize("T", [1, 2, 3, 4, 5, 8])
def test_group_law_is_dihedral(d, T):
    G = 2 * T
    r, s = (1 % T), T          # storage indices of r = (1, 0) and s = (0, 1)
    assert _power(d, r, T, T) == 0
    assert _power(d, s, 2, T) == 0
    assert d.mul(d.mul(s, r, T), s, T) == d.inv(r, T)
    for m in range(2):
        for t in range(T):
            assert d.mul(_power(d, r, t, T), _power(d, s, m, T), T) == m * T + t
    for a in range(G):
        assert d.mul(a, 0, T) == a and d.mul(0, a, T) == a
        assert d.mul(a, d.inv(a, T), T) == 0 and d.mul(d.inv(a, T), a, T) == 0
        for b in range(G):
            for c in range(G):
                assert d.mul(d.mul(a, b, T), c, T) == d.mul(a, d.mul(b, c, T), T)
    if T >= 3:
        assert d.mul(r, s, T) != d.mul(s, r, T)


def _translate(d, z, u, T):
    """(L_u z)(h) = z(u^-1 h) along the last axis."""
    G = 2 * T
    ui = d.inv(u, T)
    idx = [d.mul(ui, h, T) for h in range(G)]
    return z[..., idx]


@pytest.mark.parametrize("T", [1, 2, 3, 4, 6])
def test_equivariance_under_every_element(d, T):
    N, Cin, Cout = 5, 3, 4
    x = _rand(1, N, Cin, 2 * T)
    W = _rand(2, 2 * T, Cout, Cin)
    b = _rand(3, Cout)
    y = d.forward(x, W, b)
    for u in range(2 * T):
        yu = d.forward(_translate(d, x, u, T), W, b)
        np.testing.assert_allclose(yu, _translate(d, y, u, T), rtol=0, atol=1e-12 * np.abs(y).max())


def test_d1_is_the_cyclic_group_of_order_two(d):
    orc = oracle.oracle()
    N, Cin, Cout = 7, 3, 5
    x, W, b, dy = _rand(4, N, Cin, 2), _rand(5, 2, Cout, Cin), _rand(6, Cout), _rand(7, N, Cout, 2)
    np.testing.assert_allclose(d.forward(x, W, b), orc.forward(x, W, b), rtol=0, atol=1e-13)
    np.testing.assert_allclose(d.backward_input(dy, W), orc.backward_input(dy, W), rtol=0, atol=1e-13)
    dWd, dbd = d.backward_weight(x, dy)
    dWc, dbc = orc.backward_weight(x, dy)
    np.testing.assert_allclose(dWd, dWc, rtol=0, atol=1e-12)
    np.testing.assert_allclose(dbd, dbc, rtol=0, atol=1e-12)


def test_d2_is_a_two_dimensional_circular_convolution(d):
    """D_2 = Z2 x Z2: y[o] = sum_c ifft2(fft2(W[:, o, c]) * fft2(x[c])) on the
    2 x 2 grid (m, t)."""
    N, Cin, Cout, T = 4, 3, 2, 2
    x, W, b = _rand(8, N, Cin, 4), _rand(9, 4, Cout, Cin), _rand(10, Cout)
    xg = x.reshape(N, Cin, 2, 2)
    Wg = W.reshape(2, 2, Cout, Cin)
    ref = np.zeros((N, Cout, 2, 2))
    for o in range(Cout):
        for c in range(Cin):
            k = np.fft.fft2(Wg[:, :, o, c])
            ref[:, o] += np.real(np.fft.ifft2(np.fft.fft2(xg[:, c], axes=(1, 2)) * k, axes=(1, 2)))
    ref += b[None, :, None, None]
    np.testing.assert_allclose(d.forward(x, W, b), ref.reshape(N, Cout, 4), rtol=0, atol=1e-12)


@pytest.mark.parametrize("T", [3, 4, 8])
def test_rotations_only_reduce_to_the_cyclic_layer(d, T):
    orc = oracle.oracle()
    N, Cin, Cout = 6, 4, 3
    x = np.zeros((N, Cin, 2 * T))
    x[:, :, :T] = _rand(11, N, Cin, T)
    W = np.zeros((2 * T, Cout, Cin))
    W[:T] = _rand(12, T, Cout, Cin)
    y = d.forward(x, W, None)
    np.testing.assert_allclose(y[:, :, :T], orc.forward(x[:, :, :T], W[:T]), rtol=0, atol=1e-12)
    assert np.all(y[:, :, T:] == 0.0)


@pytest.mark.parametrize("T", [1, 3, 4, 7])
def test_gradients_are_adjoints(d, T):
    N, Cin, Cout = 6, 3, 5
    x, W, dy = _rand(13, N, Cin, 2 * T), _rand(14, 2 * T, Cout, Cin), _rand(15, N, Cout, 2 * T)
    y = d.forward(x, W, None)
    dx = d.backward_input(dy, W)
    dW, db = d.backward_weight(x, dy)
    lhs = float(np.sum(y * dy))
    assert abs(lhs - float(np.sum(x * dx))) <= 1e-11 * max(1.0, abs(lhs))
    assert abs(lhs - float(np.sum(W * dW))) <= 1e-11 * max(1.0, abs(lhs))
    np.testing.assert_allclose(db, dy.sum(axis=(0, 2)), rtol=0, atol=1e-12)


def _pins_pass(lib_path):
    """Run the pins above against one compiled copy; True if all hold."""
    try:
        dd = oracle.DihedralOracle(oracle.load_dihedral(lib_path))
        for T in (1, 2, 3, 4):
            test_group_law_is_dihedral(dd, T)
        for T in (1, 2, 3, 4):
            test_equivariance_under_every_element(dd, T)
        test_d1_is_the_cyclic_group_of_order_two(dd)
        test_d2_is_a_two_dimensional_circular_convolution(dd)
        for T in (3, 4):
            test_rotations_only_reduce_to_the_cyclic_layer(dd, T)
        for T in (1, 3, 4):
            test_gradients_are_adjoints(dd, T)
    except AssertionError:
        return False
    return True


MUTANTS = [
    ("reflection does not reverse the rotation", "int t = ma ? ta - tb : ta + tb;", "int t = ta + tb;"),
    ("inverse of a reflection negated", "int t = ma ? ta : (T - ta) % T;", "int t = (T - ta) % T;"),
    ("g h^-1 in place of h^-1 g", "const int u = d_mul(d_inv(h, T), g, T);",
     "const int u = d_mul(g, d_inv(h, T), T);"),
    ("input gradient with h^-1 g taken as g^-1 h", "const int u = d_mul(hi, g, T);",
     "const int u = d_mul(d_inv(g, T), h, T);"),
    ("weight gradient over u h in place of h u",
     "dy[(n * Cout + o) * G + d_mul(h, u, T)]", "dy[(n * Cout + o) * G + d_mul(u, h, T)]"),
    ("bias dropped", "if (b) acc += b[o];", ""),
]


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
@pytest.mark.parametrize("what,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_planted_mistakes_are_caught(what, old, new):
    src = open(SRC).read()
    assert old in src, what
    tmp = tempfile.mkdtemp()
    path = os.path.join(tmp, "mut.c")
    with open(path, "w") as f:
        f.write(src.replace(old, new, 1))
    out = os.path.join(tmp, "libmut.so")
    oracle.build(path, out)
    if what == "bias dropped":
        # the bias only shows against a reference that has one
        dd = oracle.DihedralOracle(oracle.load_dihedral(out))
        N, Cin, Cout, T = 3, 2, 2, 1
        x, W, b = _rand(20, N, Cin, 2), _rand(21, 2, Cout, Cin), _rand(22, Cout)
        with pytest.raises(AssertionError):
            np.testing.assert_allclose(dd.forward(x, W, b), oracle.oracle().forward(x, W, b),
                                       rtol=0, atol=1e-13)
        return
    assert not _pins_pass(out), what


def test_clean_copy_passes_the_mutant_harness():
    oracle.load_dihedral()
    assert _pins_pass(oracle._DLIB_PATH)
