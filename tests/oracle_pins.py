"""Pins that tie the fp64 oracle to the paper and to mathematics outside itself.

Each pin is a function taking an ``oracle.Oracle`` and raising AssertionError on
failure.  They are collected by ``test_oracle_pins.py`` for the real oracle and
re-run by ``test_oracle_mutants.py`` against deliberately broken copies of the
oracle source, to show that a plausible slip (a wrong lag sign, a dropped term,
a transposed operand) is caught by at least one of them.

What each pin is anchored to:
  * ``pin_fft_convolution_theorem`` -- numpy's FFT: the convolution theorem
    along the group axis (Sec. 3.1, Eq. 3) evaluated with ``numpy.fft``.
  * ``pin_p4_closed_form`` -- the p4 matrices printed in Sec. 3.2.2 (Step 1 and
    Step 4) and the kernel products of Appendix A.2, read from
    ``golden/p4_transforms.txt``.
  * ``pin_dense_unrolled`` -- the naive EQ-Linear: the block-circulant matrix
    assembled explicitly and applied by a dense matmul (Sec. 3.1, Eq. 1).
  * ``pin_linear_layer_T1`` / ``pin_T2_hadamard`` -- special cases that reduce
    to a plain matmul and to the 2-point DFT.
  * ``pin_roll_equivariance`` -- f(G x) = G f(x) (Sec. 4.3, the equivariance
    test of Table 5), bit-exact for the forward pass.
  * ``pin_one_hot`` -- impulse responses and the bias-only case.
  * ``pin_finite_differences`` -- L = <dy, y> is affine in each argument, so a
    central difference with step 1 is exact up to rounding.
  * ``pin_adjointness`` -- <dy, y - b> = <dx, x> = <dw, w>, and db = sum dy.
  * ``pin_entries`` -- sampled weight-gradient entries agree with the full one.
"""
from __future__ import annotations

import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")
TS = (1, 2, 3, 4, 5, 6, 8, 12, 16)


def read_matrices(path):
    mats, cur, rows = {}, None, []
    with open(path) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            if line.startswith("["):
                if cur is not None:
                    mats[cur] = np.array(rows, dtype=np.float64)
                cur, rows = line.strip("[]"), []
            else:
                rows.append([float(v) for v in line.split()])
    if cur is not None:
        mats[cur] = np.array(rows, dtype=np.float64)
    return mats


def _rand(shape, rs):
    return rs.standard_normal(shape)


def _case(T, Cin, Cout, N, seed, bias=True):
    rs = np.random.RandomState(seed)
    x = _rand((N, Cin, T), rs)
    w = _rand((T, Cout, Cin), rs)
    b = _rand((Cout,), rs) if bias else None
    dy = _rand((N, Cout, T), rs)
    return x, w, b, dy


def _rel(a, b):
    scale = max(np.max(np.abs(b)), 1e-300)
    return float(np.max(np.abs(a - b)) / scale)


# ----------------------------------------------------------------------------
def pin_fft_convolution_theorem(orc):
    """irfft( sum_c rfft_lag(w) * rfft_t(x) ) + b equals the oracle's forward,
    and the spectral gradient formulas (conjugated spectra) equal its dx, dw."""
    for i, T in enumerate(TS):
        x, w, b, dy = _case(T, 5, 7, 6, 100 + i)
        X = np.fft.fft(x, axis=2)                  # [N, Cin, T]
        W = np.fft.fft(w, axis=0)                  # [T, Cout, Cin]
        Yh = np.einsum("koc,nck->nok", W, X)
        y_fft = np.real(np.fft.ifft(Yh, axis=2)) + b[None, :, None]
        assert _rel(orc.forward(x, w, b), y_fft) < 1e-12, ("fwd", T)
        D = np.fft.fft(dy, axis=2)
        dXh = np.einsum("nok,koc->nck", D, np.conj(W))
        dx_fft = np.real(np.fft.ifft(dXh, axis=2))
        assert _rel(orc.backward_input(dy, w), dx_fft) < 1e-12, ("dx", T)
        H = np.einsum("nck,nok->koc", np.conj(X), D)   # [T, Cout, Cin]
        dw_fft = np.real(np.fft.ifft(H, axis=0))
        dw, db = orc.backward_weight(x, dy)
        assert _rel(dw, dw_fft) < 1e-12, ("dw", T)
        assert _rel(db, np.real(D[:, :, 0]).sum(0)) < 1e-12, ("db", T)


def pin_p4_closed_form(orc):
    """T = 4 through the printed p4 matrices: f = DFT4_real x, planes of w by the
    same transform over the lag, a0..a3 by the Appendix A.2 products, y by
    IDFT4_real.  Also checks the transcription against numpy's DFT."""
    m = read_matrices(os.path.join(GOLDEN, "p4_transforms.txt"))
    F = m["F4_re"] + 1j * m["F4_im"]
    assert np.allclose(F, np.fft.fft(np.eye(4), axis=0))
    Fi = m["IDFT4_re"] + 1j * m["IDFT4_im"]
    assert np.allclose(Fi, np.fft.ifft(np.eye(4), axis=0))
    R, G = m["DFT4_real"], m["IDFT4_real"]
    x, w, b, _ = _case(4, 6, 5, 7, 7)
    f = np.einsum("pt,nct->pnc", R, x)          # f0..f3 per (n, c)
    wp = np.einsum("pj,joc->poc", R, w)         # w0..w3 per (o, c)
    a0 = np.einsum("nc,oc->no", f[0], wp[0])
    a1 = np.einsum("nc,oc->no", f[1], wp[1]) - np.einsum("nc,oc->no", f[3], wp[3])
    a2 = np.einsum("nc,oc->no", f[2], wp[2])
    a3 = np.einsum("nc,oc->no", f[1], wp[3]) + np.einsum("nc,oc->no", f[3], wp[1])
    a = np.stack([a0, a1, a2, a3])              # [4, N, Cout]
    y = np.einsum("tp,pno->not", G, a) + b[None, :, None]
    assert _rel(orc.forward(x, w, b), y) < 1e-13


def _dense(w):
    """Block-circulant matrix of Eq. 1 in the convolution lag direction:
    row (o, t), column (c, s) holds w[(t - s) mod T, o, c]."""
    T, Cout, Cin = w.shape
    Wd = np.zeros((Cout * T, Cin * T))
    for t in range(T):
        for s in range(T):
            Wd[t::T, s::T] = w[(t - s) % T]
    return Wd


def pin_dense_unrolled(orc):
    for i, T in enumerate(TS):
        x, w, b, dy = _case(T, 3, 5, 4, 200 + i)
        Wd = _dense(w)
        N = x.shape[0]
        y = (x.reshape(N, -1) @ Wd.T).reshape(N, 5, T) + b[None, :, None]
        assert _rel(orc.forward(x, w, b), y) < 1e-12, ("fwd", T)
        dx = (dy.reshape(N, -1) @ Wd).reshape(x.shape)
        assert _rel(orc.backward_input(dy, w), dx) < 1e-12, ("dx", T)
        # weight tying: dw[j,o,c] = sum over the dense entries that hold w[j,o,c]
        Gd = dy.reshape(N, -1).T @ x.reshape(N, -1)          # dL/dW_dense
        dw_ref = np.zeros_like(w)
        for t in range(T):
            for s in range(T):
                dw_ref[(t - s) % T] += Gd[t::T, s::T]
        dw, db = orc.backward_weight(x, dy)
        assert _rel(dw, dw_ref) < 1e-12, ("dw", T)


def pin_linear_layer_T1(orc):
    x, w, b, dy = _case(1, 9, 6, 11, 3)
    y = x[:, :, 0] @ w[0].T + b
    assert _rel(orc.forward(x, w, b)[:, :, 0], y) < 1e-13
    assert _rel(orc.backward_input(dy, w)[:, :, 0], dy[:, :, 0] @ w[0]) < 1e-13
    dw, db = orc.backward_weight(x, dy)
    assert _rel(dw[0], dy[:, :, 0].T @ x[:, :, 0]) < 1e-13
    assert _rel(db, dy[:, :, 0].sum(0)) < 1e-13


def pin_T2_hadamard(orc):
    """T = 2: the DFT is [[1,1],[1,-1]], both bins real; y = H^-1 ((H w) * (H x))."""
    x, w, b, _ = _case(2, 4, 3, 5, 4)
    Hm = np.array([[1.0, 1.0], [1.0, -1.0]])
    xs = np.einsum("kt,nct->knc", Hm, x)
    ws = np.einsum("kj,joc->koc", Hm, w)
    ys = np.einsum("knc,koc->kno", xs, ws)
    y = np.einsum("tk,kno->not", np.linalg.inv(Hm), ys) + b[None, :, None]
    assert _rel(orc.forward(x, w, b), y) < 1e-13


def pin_roll_equivariance(orc):
    for i, T in enumerate(TS):
        x, w, b, dy = _case(T, 4, 3, 5, 300 + i)
        y = orc.forward(x, w, b)
        dx = orc.backward_input(dy, w)
        dw, _ = orc.backward_weight(x, dy)
        for r in range(T):
            assert np.array_equal(orc.forward(np.roll(x, r, axis=2), w, b),
                                  np.roll(y, r, axis=2)), ("fwd", T, r)
            assert np.array_equal(orc.backward_input(np.roll(dy, r, axis=2), w),
                                  np.roll(dx, r, axis=2)), ("dx", T, r)
            dw_r, _ = orc.backward_weight(np.roll(x, r, axis=2), np.roll(dy, r, axis=2))
            assert _rel(dw_r, dw) < 1e-13, ("dw", T, r)


def pin_one_hot(orc):
    for T in (3, 4, 8):
        rs = np.random.RandomState(T)
        Cin, Cout, N = 3, 4, 3
        w = rs.standard_normal((T, Cout, Cin))
        b = rs.standard_normal(Cout)
        # impulse input: y[n0, o, t] = w[(t - s0) mod T, o, c0] (no bias)
        n0, c0, s0 = 1, 2, T - 1
        x = np.zeros((N, Cin, T))
        x[n0, c0, s0] = 1.0
        y = orc.forward(x, w, None)
        ref = np.zeros((N, Cout, T))
        for t in range(T):
            ref[n0, :, t] = w[(t - s0) % T, :, c0]
        assert np.array_equal(y, ref), ("impulse x", T)
        # impulse weight: a cyclic shift of channel c0 by +j0 into output o0
        j0, o0 = 1, 3
        wi = np.zeros((T, Cout, Cin))
        wi[j0, o0, c0] = 1.0
        x = rs.standard_normal((N, Cin, T))
        y = orc.forward(x, wi, None)
        ref = np.zeros((N, Cout, T))
        ref[:, o0, :] = np.roll(x[:, c0, :], j0, axis=1)
        assert np.array_equal(y, ref), ("impulse w", T)
        # bias only
        y = orc.forward(np.zeros((N, Cin, T)), w, b)
        assert np.array_equal(y, np.broadcast_to(b[None, :, None], y.shape)), ("bias", T)


def pin_finite_differences(orc):
    """Central differences with h = 1 on every entry of x, w and b."""
    for i, T in enumerate((1, 2, 3, 4, 5, 8)):
        x, w, b, dy = _case(T, 3, 2, 2, 400 + i)

        def L(x_, w_, b_):
            return float(np.sum(dy * orc.forward(x_, w_, b_)))

        def fd(arr, which):
            g = np.zeros_like(arr)
            for idx in np.ndindex(arr.shape):
                p, m = arr.copy(), arr.copy()
                p[idx] += 1.0
                m[idx] -= 1.0
                args_p = {"x": (p, w, b), "w": (x, p, b), "b": (x, w, p)}[which]
                args_m = {"x": (m, w, b), "w": (x, m, b), "b": (x, w, m)}[which]
                g[idx] = 0.5 * (L(*args_p) - L(*args_m))
            return g

        dx = orc.backward_input(dy, w)
        dw, db = orc.backward_weight(x, dy)
        assert np.max(np.abs(fd(x, "x") - dx)) < 1e-10, ("dx", T)
        assert np.max(np.abs(fd(w, "w") - dw)) < 1e-10, ("dw", T)
        assert np.max(np.abs(fd(b, "b") - db)) < 1e-10, ("db", T)


def pin_adjointness(orc):
    for i, T in enumerate(TS):
        x, w, b, dy = _case(T, 6, 4, 9, 500 + i)
        y0 = orc.forward(x, w, None)
        dx = orc.backward_input(dy, w)
        dw, db = orc.backward_weight(x, dy)
        s_y = float(np.sum(dy * y0))
        assert abs(s_y - float(np.sum(dx * x))) < 1e-11 * max(1.0, abs(s_y)), ("<dx,x>", T)
        assert abs(s_y - float(np.sum(dw * w))) < 1e-11 * max(1.0, abs(s_y)), ("<dw,w>", T)
        assert _rel(db, dy.sum(axis=(0, 2))) < 1e-13, ("db", T)
        yb = orc.forward(x, w, b)
        assert _rel(yb - y0, np.broadcast_to(b[None, :, None], yb.shape)) < 1e-12


def pin_entries(orc):
    for i, T in enumerate((3, 4, 8)):
        x, w, b, dy = _case(T, 5, 6, 13, 600 + i)
        dw, _ = orc.backward_weight(x, dy)
        rs = np.random.RandomState(T)
        j = rs.randint(0, T, 20)
        o = rs.randint(0, 6, 20)
        c = rs.randint(0, 5, 20)
        assert np.array_equal(orc.backward_weight_entries(x, dy, j, o, c), dw[j, o, c]), T


ALL_PINS = [pin_fft_convolution_theorem, pin_p4_closed_form, pin_dense_unrolled,
            pin_linear_layer_T1, pin_T2_hadamard, pin_roll_equivariance, pin_one_hot,
            pin_finite_differences, pin_adjointness, pin_entries]
