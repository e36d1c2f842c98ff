"""GPU parity of the dihedral-group layer (paper_2607_21271_amd/dihedral.py:
weight expansion, the C_T kernels at 2Cin -> 2Cout channels, gradient fold)
against the fp64 D_T oracle (oracle/eqref_dihedral.c), through the C ABI.

Bar as for the C_T layer: per output tensor max|gpu - oracle| / max|oracle|
<= 1e-5 (fp32), <= 5e-3 (fp16), on the dtype-rounded inputs.
"""
import numpy as np
import pytest

import oracle
import synth
from gpu_util import TOL, rel_err, say, to_dev

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


@pytest.fixture(scope="module")
def dorc():
    return oracle.dihedral_oracle()


def _draw(T, Cin, Cout, N, bias, seed, dt):
    """x [N,Cin,2T], W [2T,Cout,Cin], b, dy drawn as the C_T workloads are
    (synth's generator at 2T group positions), rounded to dt."""
    inp = synth.draw(2 * T, Cin, Cout, N, bias, seed).rounded(dt)
    return inp.x, inp.w, inp.b, inp.dy


def _gpu(x, W, b, dy, dt, fused_env, monkeypatch):
    from paper_2607_21271_amd import dihedral
    if fused_env is None:
        monkeypatch.delenv("EQL_BWD_FUSED", raising=False)
    else:
        monkeypatch.setenv("EQL_BWD_FUSED", fused_env)
    xt = to_dev(x, dt).requires_grad_(True)
    Wt = to_dev(W, dt).requires_grad_(True)
    bt = to_dev(b, dt).requires_grad_(True) if b is not None else None
    y = dihedral.DihedralEQLinearFunction.apply(xt, Wt, bt)
    y.backward(to_dev(dy, dt))
    torch.cuda.synchronize()
    f = lambda t: None if t is None else t.detach().float().cpu().numpy()
    return {"y": f(y), "dx": f(xt.grad), "dW": f(Wt.grad), "db": f(bt.grad) if bt is not None else None}


CASES = [(1, 3, 5, 37, True), (2, 8, 8, 300, True), (3, 12, 20, 517, False), (4, 12, 48, 1037, True),
         (4, 24, 96, 333, False), (5, 7, 9, 129, True), (8, 48, 192, 257, False), (8, 16, 16, 100, True),
         (6, 20, 10, 64, True)]


@pytest.mark.parametrize("dt", ["f32", "f16"])
@pytest.mark.parametrize("T,Cin,Cout,N,bias", CASES, ids=["D%d-%dx%d-N%d" % c[:4] for c in CASES])
@pytest.mark.parametrize("path", ["auto", "fused"])
def test_dihedral_layer_matches_oracle(dorc, monkeypatch, T, Cin, Cout, N, bias, dt, path):
    """path "fused" forces the single-pass backward where a variant holds the
    C_T layer (else the two kernels run, as in "auto")."""
    say("dihedral", T, Cin, Cout, N, bias, dt, path)
    x, W, b, dy = _draw(T, Cin, Cout, N, bias, 7100 + 13 * T + Cin + 3 * Cout + N, dt)
    g = _gpu(x, W, b, dy, dt, "1" if path == "fused" else None, monkeypatch)
    y = dorc.forward(x, W, b)
    dx = dorc.backward_input(dy, W)
    dW, db = dorc.backward_weight(x, dy, with_bias=b is not None)
    errs = {"y": rel_err(g["y"], y), "dx": rel_err(g["dx"], dx), "dW": rel_err(g["dW"], dW)}
    if db is not None:
        errs["db"] = rel_err(g["db"], db)
    say("D%d %dx%d N%d" % (T, Cin, Cout, N), dt, path, {k: "%.2e" % v for k, v in errs.items()})
    for k, v in errs.items():
        assert v <= TOL[dt], (k, v)


@pytest.mark.parametrize("dt", ["f32", "f16"])
def test_dihedral_layer_is_equivariant_on_gpu(dorc, monkeypatch, dt):
    """Translating the input by every element of D_4 translates the GPU output
    (to the dtype's rounding)."""
    from paper_2607_21271_amd import dihedral
    T, Cin, Cout, N = 4, 12, 20, 200
    x, W, b, _ = _draw(T, Cin, Cout, N, True, 7301, dt)
    xt, Wt, bt = to_dev(x, dt), to_dev(W, dt), to_dev(b, dt)
    with torch.no_grad():
        y = dihedral.DihedralEQLinearFunction.apply(xt, Wt, bt).float().cpu().numpy()
        for u in range(2 * T):
            ui = dorc.inv(u, T)
            idx = [dorc.mul(ui, h, T) for h in range(2 * T)]
            yu = dihedral.DihedralEQLinearFunction.apply(xt[..., idx].contiguous(), Wt, bt)
            err = rel_err(yu.float().cpu().numpy(), y[..., idx])
            assert err <= TOL[dt], (u, err)


def test_expand_and_fold_are_adjoint(monkeypatch):
    """<expand(W), V> = <W, fold(V)> for the weights (each W entry appears at
    exactly the two places of the C_T weight that fold sums), in fp32."""
    from paper_2607_21271_amd import dihedral
    rs = np.random.RandomState(5)
    for T, Cin, Cout in ((1, 3, 2), (3, 5, 7), (8, 4, 6)):
        W = torch.from_numpy(rs.standard_normal((2 * T, Cout, Cin))).float().cuda()
        b = torch.from_numpy(rs.standard_normal(Cout)).float().cuda()
        V = torch.from_numpy(rs.standard_normal((T, 2 * Cout, 2 * Cin))).float().cuda()
        vb = torch.from_numpy(rs.standard_normal(2 * Cout)).float().cuda()
        w_ct, b_ct = dihedral.expand(W, b)
        dW, db = dihedral.fold(V, vb)
        torch.cuda.synchronize()
        lhs = float((w_ct.double() * V.double()).sum() + (b_ct.double() * vb.double()).sum())
        rhs = float((W.double() * dW.double()).sum() + (b.double() * db.double()).sum())
        assert abs(lhs - rhs) <= 1e-5 * max(1.0, abs(lhs)), (T, lhs, rhs)
        # every C_T weight entry is a copy of a W entry
        vals = set(np.round(W.cpu().numpy().ravel(), 7))
        assert set(np.round(w_ct.cpu().numpy().ravel(), 7)) <= vals
