"""GPU parity of the bfloat16 path (EQL_BF16) against the fp64 oracle, through
the C ABI.

bf16 shares every shape, layout and kernel tile with fp16; its forward
transforms run in fp32 and each spectrum value is rounded once to bf16 as an
MFMA operand (the packed fp16 transform arithmetic would lose too much at 8
significand bits); the single-pass backward is not built for bf16.  Bar, per
output tensor: max|gpu - oracle| / max|oracle| <= 4e-2, the fp16 bar of 5e-3
scaled by the ratio of the unit roundoffs (2^-8 / 2^-11 = 8), with the oracle
fed the same bf16-rounded inputs.
"""
import numpy as np
import pytest

import synth
from gpu_util import TOL, rel_err, run_gpu, say, to_dev

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

DT = "bf16"


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _check_all(inp, orc, tag):
    g = run_gpu(inp, DT)
    errs = {"y": rel_err(g["y"], orc.forward(inp.x, inp.w, inp.b)),
            "dx": rel_err(g["dx"], orc.backward_input(inp.dy, inp.w))}
    dw, db = orc.backward_weight(inp.x, inp.dy, with_bias=inp.b is not None)
    errs["dw"] = rel_err(g["dw"], dw)
    if db is not None:
        errs["db"] = rel_err(g["db"], db)
    say(tag, DT, {k: "%.2e" % v for k, v in errs.items()})
    for k, v in errs.items():
        assert v <= TOL[DT], (tag, k, v)
    return g


REDUCED_N = {"tiny_c4": 256, "vit_s_proj": 1037, "vit_b_mlp_up": 517, "vit_b_mlp_down": 517,
             "swin_s1": 2085, "sweep_T3": 1029, "sweep_T5": 1029, "sweep_T12": 1029,
             "sweep_T16": 1029}


@pytest.mark.parametrize("name", list(synth.LAYERS))
def test_layer_reduced_rows(orc, name):
    l = synth.LAYERS[name]
    say("case", name, DT, "N =", REDUCED_N[name])
    inp = synth.draw(l.T, l.Cin, l.Cout, REDUCED_N[name], l.bias, l.seed).rounded(DT)
    _check_all(inp, orc, name)


@pytest.mark.parametrize("name", ["vit_b_mlp_up", "vit_b_mlp_down", "swin_s1", "sweep_T5"])
def test_layer_full_size(orc, name):
    """Every element of y, dx, dw and db at the full workload size."""
    l = synth.LAYERS[name]
    say("case full", name, DT, "N =", l.N)
    _check_all(synth.draw_layer(l).rounded(DT), orc, name + " full")


EDGE = [(T, 5, 7, 37, True) for T in range(1, 17)] + [(T, 33, 19, 70, False) for T in range(1, 17)]
EDGE += [(8, 96, 384, 1, False), (8, 384, 96, 33, False), (12, 64, 1, 63, True), (2, 129, 130, 31, True)]


@pytest.mark.parametrize("T,Cin,Cout,N,bias", EDGE,
                         ids=["T%d-%dx%d-N%d%s" % (e[0], e[1], e[2], e[3], "-b" if e[4] else "") for e in EDGE])
def test_edge_shapes(orc, T, Cin, Cout, N, bias):
    say("edge", T, Cin, Cout, N, bias, DT)
    inp = synth.draw(T, Cin, Cout, N, bias, 9500 + 97 * T + Cin + 7 * Cout + N).rounded(DT)
    _check_all(inp, orc, "edge T%d %dx%d N%d" % (T, Cin, Cout, N))


MODES = [(3, 64, 64, 1029, True), (4, 24, 96, 2085, False), (8, 48, 48, 613, True),
         (12, 64, 64, 257, True), (8, 96, 384, 300, False)]


@pytest.mark.parametrize("mode", ["0", "1", "2"])
@pytest.mark.parametrize("T,Cin,Cout,N,bias", MODES, ids=["T%d-%dx%d-N%d" % f[:4] for f in MODES])
def test_forced_weight_mode(orc, monkeypatch, T, Cin, Cout, N, bias, mode):
    """Streamed (0), resident-spectrum (1, where the plan allows it) and
    resident-weight (2, where the blocks fit) instantiations."""
    say("forced mode", mode, T, Cin, Cout, N, DT)
    monkeypatch.setenv("EQL_GEMM_MODE", mode)
    inp = synth.draw(T, Cin, Cout, N, bias, 7100 + 31 * T + Cin + Cout).rounded(DT)
    g = run_gpu(inp, DT, want=("y", "dx"))
    errs = {"y": rel_err(g["y"], orc.forward(inp.x, inp.w, inp.b)),
            "dx": rel_err(g["dx"], orc.backward_input(inp.dy, inp.w))}
    say("  ", {k: "%.2e" % v for k, v in errs.items()})
    for k, v in errs.items():
        assert v <= TOL[DT], (T, Cin, Cout, mode, k, v)


KIND_CASES = [(8, 96, 384, 700, False), (4, 24, 96, 1111, False), (3, 64, 64, 517, True),
              (16, 40, 24, 300, True), (4, 512, 512, 260, True), (5, 7, 33, 129, True)]


@pytest.mark.parametrize("kind", ["0", "1"])
@pytest.mark.parametrize("T,Cin,Cout,N,bias", KIND_CASES, ids=["T%d-%dx%d-N%d" % f[:4] for f in KIND_CASES])
def test_weight_gradient_kernels(orc, monkeypatch, T, Cin, Cout, N, bias, kind):
    """Both weight-gradient kernels in bf16: staged (0) and register-direct (1),
    each summing the bias from the fp32 bin 0."""
    say("wgrad kind", kind, T, Cin, Cout, N, DT)
    monkeypatch.setenv("EQL_WGRAD_KIND", kind)
    inp = synth.draw(T, Cin, Cout, N, bias, 7300 + 31 * T + Cin + Cout).rounded(DT)
    g = run_gpu(inp, DT, want=("dw",))
    dw, db = orc.backward_weight(inp.x, inp.dy, with_bias=bias)
    errs = {"dw": rel_err(g["dw"], dw)}
    if bias:
        errs["db"] = rel_err(g["db"], db)
    say("  ", {k: "%.2e" % v for k, v in errs.items()})
    for k, v in errs.items():
        assert v <= TOL[DT], (T, Cin, Cout, kind, k, v)


def test_zero_rows():
    from paper_2607_21271_amd import ops
    T, Cin, Cout = 8, 16, 24
    w = to_dev(np.random.RandomState(1).standard_normal((T, Cout, Cin)), DT)
    b = to_dev(np.ones(Cout), DT)
    wspec = ops.weight_spectrum(w)
    x = torch.empty(0, Cin, T, dtype=w.dtype, device="cuda")
    y = ops.forward(x, wspec, b, T, Cin, Cout)
    dw = torch.full((T, Cout, Cin), 7.0, dtype=w.dtype, device="cuda")
    db = torch.full((Cout,), 7.0, dtype=w.dtype, device="cuda")
    ops.backward_weight(x, torch.empty(0, Cout, T, dtype=w.dtype, device="cuda"), T, Cin, Cout,
                        True, dw=dw, db=db)
    torch.cuda.synchronize()
    assert y.shape == (0, Cout, T)
    assert torch.all(dw == 0) and torch.all(db == 0)


def test_bitwise_determinism_and_whole_backward():
    """Two runs agree bit for bit, and eqlinear_backward (always two passes for
    bf16) equals the separate input- and weight-gradient calls bit for bit."""
    from paper_2607_21271_amd import ops
    l = synth.LAYERS["vit_b_mlp_up"].with_n(3001)
    inp = synth.draw(l.T, l.Cin, l.Cout, l.N, True, l.seed).rounded(DT)
    a, b = run_gpu(inp, DT), run_gpu(inp, DT)
    for k in a:
        assert np.array_equal(a[k], b[k]), k
    assert not ops.backward_is_fused(l.N, l.T, l.Cin, l.Cout, torch.bfloat16)
    x, w, dy = to_dev(inp.x, DT), to_dev(inp.w, DT), to_dev(inp.dy, DT)
    wspec = ops.weight_spectrum(w)
    dx, dw, db = ops.backward(x, dy, wspec, l.T, l.Cin, l.Cout, with_bias=True)
    torch.cuda.synchronize()
    assert np.array_equal(dx.float().cpu().numpy(), a["dx"])
    assert np.array_equal(dw.float().cpu().numpy(), a["dw"])
    assert np.array_equal(db.float().cpu().numpy(), a["db"])


def test_output_rounding_is_nearest_even():
    """T = 1, two input channels, unit weights: y = x0 + x1 is exact in the
    fp32 accumulator and rounded once to bf16.  Sums at and beside the halfway
    points between bf16 neighbours come out as round-to-nearest-even."""
    from paper_2607_21271_amd import ops
    u = 2.0 ** -8   # half an ulp of bf16 at 1.0
    pairs = [(1.0, u), (1.0, 3 * u), (1.0, 5 * u), (-1.0, -u), (1.0, u * 1.5), (2.0, 2 * u), (1.0, -u / 2)]
    x0 = np.array([p[0] for p in pairs])
    x1 = np.array([p[1] for p in pairs])
    assert np.array_equal(synth.round_to(x1, DT), x1) and np.array_equal(synth.round_to(x0, DT), x0)
    N = len(pairs)
    x = to_dev(np.stack([x0, x1], axis=1).reshape(N, 2, 1), DT)
    w = to_dev(np.ones((1, 1, 2)), DT)
    y = ops.forward(x, ops.weight_spectrum(w), None, 1, 2, 1).float().cpu().numpy().reshape(N)
    exact = x0 + x1                       # exact in float64 and in fp32
    want = torch.tensor(exact, dtype=torch.float32).to(torch.bfloat16).float().numpy()
    say("rounding", list(zip(exact.tolist(), y.tolist())))
    assert np.array_equal(y, want), (y, want)
    assert y[0] == 1.0 and y[1] == 1.0 + 4 * u and y[2] == 1.0 + 4 * u   # ties to even


def test_autograd_module_matches_oracle(orc):
    from paper_2607_21271_amd.ops import EQLinear
    T, Cin, Cout, N = 8, 24, 40, 130
    inp = synth.draw(T, Cin, Cout, N, True, 4343).rounded(DT)
    m = EQLinear(T, Cin, Cout, bias=True, device="cuda", dtype=torch.bfloat16)
    with torch.no_grad():
        m.weight.copy_(to_dev(inp.w, DT))
        m.bias.copy_(to_dev(inp.b, DT))
    x = to_dev(inp.x, DT).view(2, 65, Cin, T).requires_grad_(True)
    y = m(x)
    y.backward(to_dev(inp.dy, DT).view(2, 65, Cout, T))
    torch.cuda.synchronize()
    ref_dw, ref_db = orc.backward_weight(inp.x, inp.dy)
    errs = {"y": rel_err(y.detach().float().cpu().numpy().reshape(N, Cout, T), orc.forward(inp.x, inp.w, inp.b)),
            "dx": rel_err(x.grad.float().cpu().numpy().reshape(N, Cin, T), orc.backward_input(inp.dy, inp.w)),
            "dw": rel_err(m.weight.grad.float().cpu().numpy(), ref_dw),
            "db": rel_err(m.bias.grad.float().cpu().numpy(), ref_db)}
    say("autograd", DT, {k: "%.2e" % v for k, v in errs.items()})
    for k, v in errs.items():
        assert v <= TOL[DT], (k, v)


def test_dihedral_layer_matches_oracle():
    """The D_T layer in bf16 (weight gather and gradient fold kernels at bf16,
    the C_T kernels at 2Cin -> 2Cout)."""
    import oracle
    from paper_2607_21271_amd import dihedral
    do = oracle.dihedral_oracle()
    for T, Cin, Cout, N, bias in ((4, 6, 10, 301, True), (8, 24, 48, 517, False), (3, 5, 7, 99, True)):
        rs = np.random.RandomState(610 + T)
        r = lambda a: synth.round_to(a, DT).astype(np.float64)
        x = r(rs.standard_normal((N, Cin, 2 * T)))
        W = r(rs.standard_normal((2 * T, Cout, Cin)) / np.sqrt(2 * T * Cin))
        b = r(0.1 * rs.standard_normal(Cout)) if bias else None
        dy = r(rs.standard_normal((N, Cout, 2 * T)))
        xt = to_dev(x, DT).requires_grad_(True)
        Wt = to_dev(W, DT).requires_grad_(True)
        bt = to_dev(b, DT).requires_grad_(True) if bias else None
        y = dihedral.DihedralEQLinearFunction.apply(xt, Wt, bt)
        y.backward(to_dev(dy, DT))
        torch.cuda.synchronize()
        ref_dW, ref_db = do.backward_weight(x, dy, with_bias=bias)
        errs = {"y": rel_err(y.detach().float().cpu().numpy(), do.forward(x, W, b)),
                "dx": rel_err(xt.grad.float().cpu().numpy(), do.backward_input(dy, W)),
                "dW": rel_err(Wt.grad.float().cpu().numpy(), ref_dW)}
        if bias:
            errs["db"] = rel_err(bt.grad.float().cpu().numpy(), ref_db)
        say("dihedral", T, Cin, Cout, N, DT, {k: "%.2e" % v for k, v in errs.items()})
        for k, v in errs.items():
            assert v <= TOL[DT], (T, k, v)


def test_group_conv_matches_oracle():
    """The group convolution in bf16 (patch gather, scatter and weight
    permutations at bf16)."""
    import oracle
    from paper_2607_21271_amd import gconv
    go = oracle.gconv_oracle()
    for B, H, W, T, Cin, Cout, k, bias in ((2, 7, 7, 4, 3, 5, 3, True), (1, 9, 6, 2, 8, 16, 5, False),
                                           (2, 6, 5, 1, 5, 7, 3, True)):
        rs = np.random.RandomState(8600 + T + k)
        r = lambda a: synth.round_to(a, DT).astype(np.float64)
        f = r(rs.standard_normal((B, H, W, Cin, T)))
        psi = r(rs.standard_normal((k, k, T, Cout, Cin)) / np.sqrt(k * k * T * Cin))
        b = r(0.1 * rs.standard_normal(Cout)) if bias else None
        dout = r(rs.standard_normal((B, H, W, Cout, T)))
        ft = to_dev(f, DT).requires_grad_(True)
        pt = to_dev(psi, DT).requires_grad_(True)
        bt = to_dev(b, DT).requires_grad_(True) if bias else None
        y = gconv.GroupConv2dFunction.apply(ft, pt, bt)
        y.backward(to_dev(dout, DT))
        torch.cuda.synchronize()
        ref_dpsi, ref_db = go.backward_weight(f, dout, k, with_bias=bias)
        errs = {"y": rel_err(y.detach().float().cpu().numpy(), go.forward(f, psi, b)),
                "df": rel_err(ft.grad.float().cpu().numpy(), go.backward_input(dout, psi)),
                "dpsi": rel_err(pt.grad.float().cpu().numpy(), ref_dpsi)}
        if bias:
            errs["db"] = rel_err(bt.grad.float().cpu().numpy(), ref_db)
        say("gconv", B, H, W, T, Cin, Cout, k, DT, {kk: "%.2e" % v for kk, v in errs.items()})
        for kk, v in errs.items():
            assert v <= TOL[DT], (T, k, kk, v)
