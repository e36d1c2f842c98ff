"""Pins of the group-convolution oracle (oracle/eqref_gconv.c) on the CPU.

The layer carries the C_T weight sharing (Sec. 3.1, Eq. 1-2) to a
convolution over the image plane that rotates its offsets with the group
element (Sec. 5 names equivariant convolutions as the next operators).  The
oracle is pinned against facts that do not come from it:

* equivariance: rotating a square image about its centre by 360/T degrees
  (numpy.rot90) and shifting the group axis by one rotates and shifts the
  output the same way (T = 4 and T = 2);
* a 1 x 1 kernel is the C_T layer (the separately pinned C_T oracle) with
  the lag read as a correlation;
* T = 1 is a plain 2-d cross-correlation with zero padding
  (torch.nn.functional.conv2d in float64);
* the gradients are the adjoints of the forward map;
* the input gradient is itself a group convolution of the output gradient,
  with the weight psi'[d][l][c][o] = psi[-R^-l d][-l mod T][o][c] (the form
  the GPU path uses for it).
Planted mistakes in copies of the source are caught by these pins.
"""
import os
import shutil
import tempfile

import numpy as np
import pytest

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(os.path.dirname(HERE), "oracle", "eqref_gconv.c")


@pytest.fixture(scope="module")
def go():
    return oracle.gconv_oracle()


def _rand(seed, *shape):
    return np.random.RandomState(seed).standard_normal(shape)


def _act(z, T, steps=1):
    """The group action on features [B, H, W, C, T]: rotate the image by
    360/T degrees per step and shift the group axis by one per step."""
    quarter = {4: 1, 2: 2, 1: 0}[T]
    z = np.rot90(z, k=quarter * steps, axes=(1, 2))
    return np.roll(z, steps, axis=-1)


@pytest.mark.parametrize("T,k,H", [(4, 3, 7), (4, 5, 6), (2, 3, 5), (4, 1, 4), (2, 5, 8)])
def test_rotation_equivariance(go, T, k, H):
    B, Cin, Cout = 2, 3, 4
    f = _rand(1, B, H, H, Cin, T)
    psi = _rand(2, k, k, T, Cout, Cin)
    b = _rand(3, Cout)
    out = go.forward(f, psi, b)
    for steps in range(1, T):
        got = go.forward(_act(f, T, steps), psi, b)
        np.testing.assert_allclose(got, _act(out, T, steps), rtol=0, atol=1e-12 * np.abs(out).max())


@pytest.mark.parametrize("T", [1, 2, 4])
def test_one_by_one_kernel_is_the_cyclic_layer(go, T):
    orc = oracle.oracle()
    B, H, W, Cin, Cout = 2, 3, 5, 4, 6
    f = _rand(4, B, H, W, Cin, T)
    psi = _rand(5, 1, 1, T, Cout, Cin)
    b = _rand(6, Cout)
    # correlation lag: out[r] = sum_s psi[(s - r) mod T] f[s] = sum_s w[(r - s) mod T] f[s]
    w = np.stack([psi[0, 0, (-j) % T] for j in range(T)])
    ref = orc.forward(f.reshape(-1, Cin, T), w, b).reshape(B, H, W, Cout, T)
    np.testing.assert_allclose(go.forward(f, psi, b), ref, rtol=0, atol=1e-12)


@pytest.mark.parametrize("k", [1, 3, 5])
def test_t1_is_a_plain_cross_correlation(go, k):
    torch = pytest.importorskip("torch")
    B, H, W, Cin, Cout = 2, 6, 7, 3, 4
    f = _rand(7, B, H, W, Cin, 1)
    psi = _rand(8, k, k, 1, Cout, Cin)
    b = _rand(9, Cout)
    x = torch.from_numpy(f[..., 0].transpose(0, 3, 1, 2).copy())          # [B, Cin, H, W]
    wt = torch.from_numpy(psi[:, :, 0].transpose(2, 3, 0, 1).copy())      # [Cout, Cin, k, k]
    ref = torch.nn.functional.conv2d(x, wt, torch.from_numpy(b), padding=k // 2).numpy()
    np.testing.assert_allclose(go.forward(f, psi, b)[..., 0], ref.transpose(0, 2, 3, 1), rtol=0, atol=1e-12)


@pytest.mark.parametrize("T,k", [(4, 3), (2, 3), (1, 3), (4, 5)])
def test_gradients_are_adjoints(go, T, k):
    B, H, W, Cin, Cout = 2, 5, 6, 3, 4
    f = _rand(10, B, H, W, Cin, T)
    psi = _rand(11, k, k, T, Cout, Cin)
    dout = _rand(12, B, H, W, Cout, T)
    out = go.forward(f, psi, None)
    df = go.backward_input(dout, psi)
    dpsi, db = go.backward_weight(f, dout, k)
    lhs = float(np.sum(out * dout))
    assert abs(lhs - float(np.sum(f * df))) <= 1e-10 * max(1.0, abs(lhs))
    assert abs(lhs - float(np.sum(psi * dpsi))) <= 1e-10 * max(1.0, abs(lhs))
    np.testing.assert_allclose(db, dout.sum(axis=(0, 1, 2, 4)), rtol=0, atol=1e-11)


def _adjoint_weight(psi, T):
    """psi'[d][l][c][o] = psi[-R^-l d][-l mod T][o][c] for psi [k, k, T, Cout,
    Cin] (offsets d = (a, b) at index (a + k//2, b + k//2); R(a, b) = (-b, a)
    at T = 4, (-a, -b) at T = 2)."""
    k = psi.shape[0]
    h = k // 2
    Cout, Cin = psi.shape[3], psi.shape[4]
    out = np.zeros((k, k, T, Cin, Cout))
    for a in range(-h, h + 1):
        for b in range(-h, h + 1):
            for l in range(T):
                ra, rb = a, b
                for _ in range((T - l) % T * (4 // T if T > 1 else 0)):   # R^-l = R^(T-l), quarter turns
                    ra, rb = -rb, ra
                out[a + h, b + h, l] = psi[-ra + h, -rb + h, (-l) % T].T
    return out


@pytest.mark.parametrize("T,k", [(4, 3), (4, 5), (2, 3), (2, 5), (1, 3), (4, 1)])
def test_input_gradient_is_the_adjoint_convolution(go, T, k):
    B, H, W, Cin, Cout = 2, 6, 5, 3, 4
    psi = _rand(20 + k, k, k, T, Cout, Cin)
    dout = _rand(21 + T, B, H, W, Cout, T)
    df = go.backward_input(dout, psi)
    via = go.forward(dout, _adjoint_weight(psi, T), None)
    np.testing.assert_allclose(via, df, rtol=0, atol=1e-12 * max(1.0, float(np.abs(df).max())))


def _pins_pass(lib_path):
    try:
        g = oracle.GconvOracle(oracle.load_gconv(lib_path))
        for T, k, H in ((4, 3, 7), (2, 3, 5)):
            test_rotation_equivariance(g, T, k, H)
        for T in (1, 2, 4):
            test_one_by_one_kernel_is_the_cyclic_layer(g, T)
        for k in (1, 3):
            test_t1_is_a_plain_cross_correlation(g, k)
        for T, k in ((4, 3), (2, 3), (1, 3)):
            test_gradients_are_adjoints(g, T, k)
    except AssertionError:
        return False
    return True


MUTANTS = [
    ("offset rotated the wrong way", "rot(-r, T, dy, dx, &ry, &rx);\n                for (int s = 0; s < T; ++s) {",
     "rot(r, T, dy, dx, &ry, &rx);\n                for (int s = 0; s < T; ++s) {"),
    ("group lag with the wrong sign", "const int l = ((s - r) % T + T) % T;\n                  for (int c = 0;",
     "const int l = ((r - s) % T + T) % T;\n                  for (int c = 0;"),
    ("bias dropped", "if (bias) acc += bias[o];", ""),
    ("circular padding in place of zeros",
     "const int yy = y + dy, xx = x + dx;\n                if (yy < 0 || yy >= H || xx < 0 || xx >= W) continue;\n                int ry",
     "const int yy = (y + dy + H) % H, xx = (x + dx + W) % W;\n                int ry"),
    ("input gradient without the rotation", "rot(-r, T, dy, dx, &ry, &rx);\n                  const int l",
     "ry = dy; rx = dx;\n                  const int l"),
    ("weight gradient offset unrotated", "rot(r, T, dy, dx, &ry, &rx);\n                    const int yy",
     "ry = dy; rx = dx;\n                    const int yy"),
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
    assert not _pins_pass(out), what


def test_clean_copy_passes_the_mutant_harness():
    oracle.load_gconv()
    assert _pins_pass(oracle._GLIB_PATH)
