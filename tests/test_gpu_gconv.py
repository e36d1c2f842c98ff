"""GPU parity of the rotation-equivariant group convolution
(paper_2607_21271_amd/gconv.py: patch gather, the C_T kernels at k*k*Cin
input channels, gather adjoint and weight permutations) against the fp64
group-convolution oracle (oracle/eqref_gconv.c), through the C ABI.

Bar as for the C_T layer: per output tensor max|gpu - oracle| / max|oracle|
<= 1e-5 (fp32), <= 5e-3 (fp16), on the dtype-rounded inputs.
"""
import numpy as np
import pytest

import oracle
from gpu_util import TOL, rel_err, say, to_dev

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


@pytest.fixture(scope="module")
def go():
    return oracle.gconv_oracle()


def _draw(B, H, W, T, Cin, Cout, k, bias, seed, dt):
    """Seeded unit-normal features and gradients, weights scaled by
    1/sqrt(k*k*T*Cin), rounded to the run dtype (the oracle gets the rounded
    values)."""
    import synth
    rs = np.random.RandomState(seed)
    rnd = lambda a: synth.round_to(a, dt).astype(np.float64)
    f = rnd(rs.standard_normal((B, H, W, Cin, T)))
    psi = rnd(rs.standard_normal((k, k, T, Cout, Cin)) / np.sqrt(k * k * T * Cin))
    b = rnd(0.1 * rs.standard_normal(Cout)) if bias else None
    dout = rnd(rs.standard_normal((B, H, W, Cout, T)))
    return f, psi, b, dout


CASES = [(2, 7, 7, 4, 3, 5, 3, True), (1, 9, 6, 4, 8, 16, 5, False), (3, 5, 8, 2, 6, 4, 3, True),
         (2, 6, 5, 1, 5, 7, 3, True), (2, 8, 8, 4, 24, 48, 3, True), (1, 4, 4, 4, 3, 2, 1, True),
         (2, 5, 5, 2, 4, 4, 7, False), (4, 16, 16, 4, 12, 24, 3, True)]


@pytest.mark.parametrize("dt", ["f32", "f16"])
@pytest.mark.parametrize("B,H,W,T,Cin,Cout,k,bias", CASES,
                         ids=["B%dx%dx%d-T%d-%dx%d-k%d" % c[:7] for c in CASES])
def test_group_conv_matches_oracle(go, B, H, W, T, Cin, Cout, k, bias, dt):
    from paper_2607_21271_amd import gconv
    say("gconv", B, H, W, T, Cin, Cout, k, bias, dt)
    f, psi, b, dout = _draw(B, H, W, T, Cin, Cout, k, bias, 8200 + 7 * T + k + Cin + Cout, dt)
    ft = to_dev(f, dt).requires_grad_(True)
    pt = to_dev(psi, dt).requires_grad_(True)
    bt = to_dev(b, dt).requires_grad_(True) if b is not None else None
    y = gconv.GroupConv2dFunction.apply(ft, pt, bt)
    y.backward(to_dev(dout, dt))
    torch.cuda.synchronize()
    ref_y = go.forward(f, psi, b)
    ref_df = go.backward_input(dout, psi)
    ref_dpsi, ref_db = go.backward_weight(f, dout, k, with_bias=b is not None)
    errs = {"y": rel_err(y.detach().float().cpu().numpy(), ref_y),
            "df": rel_err(ft.grad.float().cpu().numpy(), ref_df),
            "dpsi": rel_err(pt.grad.float().cpu().numpy(), ref_dpsi)}
    if b is not None:
        errs["db"] = rel_err(bt.grad.float().cpu().numpy(), ref_db)
    say("  ", {kk: "%.2e" % v for kk, v in errs.items()})
    for kk, v in errs.items():
        assert v <= TOL[dt], (kk, v)


@pytest.mark.parametrize("dt", ["f32", "f16"])
@pytest.mark.parametrize("T", [4, 2])
@pytest.mark.parametrize("Cin", [6, 8])
def test_group_conv_is_equivariant_on_gpu(dt, T, Cin):
    """Rotating the image about its centre by 360/T degrees and shifting the
    group axis by one rotates and shifts the GPU output the same way (to the
    dtype's rounding); Cin = 8 takes the implicit-gather forward."""
    from paper_2607_21271_amd import gconv
    B, H, Cout, k = 2, 9, 8, 3
    f, psi, b, _ = _draw(B, H, H, T, Cin, Cout, k, True, 8400 + T, dt)
    quarter = 1 if T == 4 else 2
    act = lambda z: np.roll(np.rot90(z, k=quarter, axes=(1, 2)), 1, axis=-1)
    with torch.no_grad():
        pt, bt = to_dev(psi, dt), to_dev(b, dt)
        y = gconv.GroupConv2dFunction.apply(to_dev(f, dt), pt, bt).float().cpu().numpy()
        yr = gconv.GroupConv2dFunction.apply(to_dev(np.ascontiguousarray(act(f)), dt), pt, bt)
        err = rel_err(yr.float().cpu().numpy(), np.ascontiguousarray(act(y)))
    say("gconv equivariance", T, dt, "%.2e" % err)
    assert err <= TOL[dt]


def test_gather_scatter_adjoint_and_weight_permutation():
    """<gather(f), V> = <f, scatter(V)>, and unpack(pack(psi)) = psi bit for
    bit (the weight map is a permutation), fp32."""
    from paper_2607_21271_amd import gconv
    rs = np.random.RandomState(3)
    for B, H, W, T, Cin, Cout, k in ((2, 5, 6, 4, 3, 2, 3), (1, 7, 7, 2, 2, 3, 5), (2, 4, 5, 1, 3, 2, 3),
                                     (1, 6, 6, 4, 2, 2, 7)):
        f = torch.from_numpy(rs.standard_normal((B, H, W, Cin, T))).float().cuda()
        V = torch.from_numpy(rs.standard_normal((B * H * W, k * k * Cin, T))).float().cuda()
        X = gconv.gather(f, T, k)
        df = gconv.scatter(V, B, H, W, T, Cin, k)
        psi = torch.from_numpy(rs.standard_normal((k, k, T, Cout, Cin))).float().cuda()
        back = gconv.unpack_weight_grad(gconv.pack_weight(psi), k)
        torch.cuda.synchronize()
        lhs = float((X.double() * V.double()).sum())
        rhs = float((f.double() * df.double()).sum())
        assert abs(lhs - rhs) <= 1e-4 * max(1.0, abs(lhs)), (T, k, lhs, rhs)
        assert torch.equal(back, psi), (T, k)


IMPLICIT = [(2, 7, 7, 4, 4, 5, 3, True), (1, 9, 6, 4, 8, 16, 5, False), (3, 5, 8, 2, 8, 4, 3, True),
            (2, 6, 5, 1, 4, 7, 3, True), (2, 8, 8, 4, 24, 48, 3, True), (1, 4, 4, 4, 4, 2, 1, True),
            (2, 5, 5, 2, 4, 4, 7, False), (4, 16, 16, 4, 12, 24, 3, True), (1, 11, 13, 4, 32, 96, 3, False)]


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("B,H,W,T,Cin,Cout,k,bias", IMPLICIT,
                         ids=["B%dx%dx%d-T%d-%dx%d-k%d" % c[:7] for c in IMPLICIT])
def test_implicit_gather_forward(go, B, H, W, T, Cin, Cout, k, bias, dt):
    """eqlinear_gconv_forward (patches read straight from f by the forward
    kernel) equals the patch gather followed by eqlinear_forward bit for bit,
    and the oracle to the dtype's bar."""
    from paper_2607_21271_amd import gconv, ops
    say("gconv implicit", B, H, W, T, Cin, Cout, k, bias, dt)
    f, psi, b, _ = _draw(B, H, W, T, Cin, Cout, k, bias, 8700 + 7 * T + k + Cin + Cout, dt)
    ft, pt = to_dev(f, dt), to_dev(psi, dt)
    bt = to_dev(b, dt) if b is not None else None
    wspec = ops.weight_spectrum(gconv.pack_weight(pt))
    y = gconv.forward_implicit(ft, wspec, bt, T, Cout, k)
    y_ref = ops.forward(gconv.gather(ft, T, k), wspec, bt, T, k * k * Cin, Cout).view(B, H, W, Cout, T)
    torch.cuda.synchronize()
    assert torch.equal(y.view(torch.int16 if dt != "f32" else torch.int32),
                       y_ref.view(torch.int16 if dt != "f32" else torch.int32))
    err = rel_err(y.float().cpu().numpy(), go.forward(f, psi, b))
    say("  ", "%.2e" % err)
    assert err <= TOL[dt]


def test_implicit_gather_refuses_unaligned_channels():
    from paper_2607_21271_amd import _lib, gconv, ops
    f = torch.zeros(1, 4, 4, 3, 4, device="cuda")
    wspec = ops.weight_spectrum(gconv.pack_weight(torch.zeros(3, 3, 4, 5, 3, device="cuda")))
    with pytest.raises(_lib.EqlError) as e:
        gconv.forward_implicit(f, wspec, None, 4, 5, 3)
    assert e.value.status == _lib.EQL_ERR_UNSUPPORTED
    assert not gconv.implicit_ok(3) and gconv.implicit_ok(8)


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("B,H,W,T,Cin,Cout,k,bias", IMPLICIT[:5],
                         ids=["B%dx%dx%d-T%d-%dx%d-k%d" % c[:7] for c in IMPLICIT[:5]])
def test_frozen_weight_group_conv(go, B, H, W, T, Cin, Cout, k, bias, dt):
    """A frozen weight (no gradient for psi or b): the autograd function runs
    the implicit-gather forward and the input gradient alone; output and
    feature gradient against the oracle."""
    from paper_2607_21271_amd import gconv
    say("gconv frozen", B, H, W, T, Cin, Cout, k, bias, dt)
    f, psi, b, dout = _draw(B, H, W, T, Cin, Cout, k, bias, 8700 + 7 * T + k + Cin, dt)
    ft = to_dev(f, dt).requires_grad_(True)
    pt = to_dev(psi, dt)
    bt = to_dev(b, dt) if b is not None else None
    y = gconv.GroupConv2dFunction.apply(ft, pt, bt)
    y.backward(to_dev(dout, dt))
    torch.cuda.synchronize()
    ey = rel_err(y.detach().float().cpu().numpy(), go.forward(f, psi, b))
    edf = rel_err(ft.grad.float().cpu().numpy(), go.backward_input(dout, psi))
    say("  y %.2e df %.2e" % (ey, edf))
    assert ey <= TOL[dt] and edf <= TOL[dt], (ey, edf)


@pytest.mark.parametrize("T,k", [(4, 3), (4, 5), (2, 3), (1, 3), (4, 1), (2, 7)])
def test_adjoint_weight_pack_is_the_permuted_pack(T, k):
    """pack_weight_adjoint(psi) equals pack_weight of the adjoint weight
    psi'[d][l][c][o] = psi[-R^-l d][-l mod T][o][c] built on the host (the
    identity pinned against the oracle on the CPU), bit for bit: both are
    permutations."""
    from paper_2607_21271_amd import gconv
    from test_gconv_oracle import _adjoint_weight
    rs = np.random.RandomState(30 + 7 * T + k)
    Cout, Cin = 5, 3
    psi = rs.standard_normal((k, k, T, Cout, Cin)).astype(np.float32)
    adj = _adjoint_weight(psi.astype(np.float64), T).astype(np.float32)
    got = gconv.pack_weight_adjoint(torch.from_numpy(psi).cuda())
    want = gconv.pack_weight(torch.from_numpy(np.ascontiguousarray(adj)).cuda())
    torch.cuda.synchronize()
    assert got.shape == (T, Cin, k * k * Cout)
    assert torch.equal(got, want)
