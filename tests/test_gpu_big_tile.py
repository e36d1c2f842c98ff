"""GPU parity of the large-tile kernels (T in {2, 4}) against the fp64 oracle,
through the C ABI: the forward / input gradient (csrc/eql_gemm_big.h: 128 x 128
output tiles) and the weight gradient (csrc/eql_wgrad_big.h: row-contiguous
spectra, 128 x 128 (c, o) tiles, row splits, the split-partial reduction), in
fp32, fp16 and bf16; fp32 at T = 4 takes three-product complex bins and
96-channel output tiles by default, EQL_GAUSS=0 the four products.

The host takes this kernel for wide layers only; EQL_GEMM_BIG=1 forces it
wherever the shape allows (contraction channels a multiple of 32), so small
shapes with ragged rows and ragged output-channel tiles cover its tails.  A
pass whose contraction channels are not a multiple of 32 keeps the other
kernel (the input gradient of the Cout = 200 case).  EQL_WGRAD_KIND=2 forces
the weight-gradient path likewise.  Bar as for the layer:
max|gpu - oracle| / max|oracle| <= 1e-5 (fp32), 5e-3 (fp16), 4e-2 (bf16).
"""
import numpy as np
import pytest

import synth
from gpu_util import TOL, rel_err, run_gpu, say, to_dev

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


CASES = [(4, 32, 128, 128, True), (4, 64, 200, 300, True), (4, 160, 96, 1000, False),
         (2, 96, 256, 777, True), (4, 512, 512, 515, True), (2, 256, 64, 129, False),
         (4, 128, 384, 1, True), (4, 1024, 160, 259, True)]


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("T,Cin,Cout,N,bias", CASES, ids=["T%d-%dx%d-N%d" % c[:4] for c in CASES])
def test_big_tile_matches_oracle(orc, monkeypatch, T, Cin, Cout, N, bias, dt):
    say("big tile", T, Cin, Cout, N, bias, dt)
    monkeypatch.setenv("EQL_GEMM_BIG", "1")
    inp = synth.draw(T, Cin, Cout, N, bias, 9100 + 13 * T + Cin + Cout).rounded(dt)
    g = run_gpu(inp, dt, want=("y", "dx"))
    errs = {"y": rel_err(g["y"], orc.forward(inp.x, inp.w, inp.b)),
            "dx": rel_err(g["dx"], orc.backward_input(inp.dy, inp.w))}
    say("  ", {k: "%.2e" % v for k, v in errs.items()})
    for k, v in errs.items():
        assert v <= TOL[dt], (k, v)


GAUSS_CASES = [(4, 32, 96, 128, True), (4, 64, 200, 300, True), (4, 160, 97, 1000, False),
               (4, 128, 384, 1, True), (4, 512, 512, 515, True), (4, 96, 1, 77, True)]


@pytest.mark.parametrize("gauss", ["0", "1"])
@pytest.mark.parametrize("T,Cin,Cout,N,bias", GAUSS_CASES, ids=["T%d-%dx%d-N%d" % c[:4] for c in GAUSS_CASES])
def test_big_tile_fp32_three_and_four_products(orc, monkeypatch, T, Cin, Cout, N, bias, gauss):
    """fp32 at T = 4 in both forms of the complex-bin product: the three
    multiplications (96-channel tiles, ragged channel tiles included) and the
    four; forward, input gradient and the large-tile weight gradient against
    the oracle."""
    say("big tile fp32 gauss", gauss, T, Cin, Cout, N, bias)
    monkeypatch.setenv("EQL_GEMM_BIG", "1")
    monkeypatch.setenv("EQL_WGRAD_KIND", "2")
    monkeypatch.setenv("EQL_GAUSS", gauss)
    inp = synth.draw(T, Cin, Cout, N, bias, 9200 + Cin + Cout + N).rounded("f32")
    g = run_gpu(inp, "f32")
    ref_dw, ref_db = orc.backward_weight(inp.x, inp.dy, with_bias=bias)
    errs = {"y": rel_err(g["y"], orc.forward(inp.x, inp.w, inp.b)),
            "dx": rel_err(g["dx"], orc.backward_input(inp.dy, inp.w)),
            "dw": rel_err(g["dw"], ref_dw)}
    if bias:
        errs["db"] = rel_err(g["db"], ref_db)
    say("  ", {k: "%.2e" % v for k, v in errs.items()})
    for k, v in errs.items():
        assert v <= TOL["f32"], (k, v)


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
def test_big_tile_same_as_default_kernel_off(orc, monkeypatch, dt):
    """The kernel switch changes no result beyond rounding: forced on and off
    agree with each other to the dtype's bar (the two kernels sum in
    different orders)."""
    T, Cin, Cout, N = 4, 256, 256, 700
    inp = synth.draw(T, Cin, Cout, N, True, 9300).rounded(dt)
    monkeypatch.setenv("EQL_GEMM_BIG", "1")
    on = run_gpu(inp, dt, want=("y", "dx"))
    monkeypatch.setenv("EQL_GEMM_BIG", "0")
    off = run_gpu(inp, dt, want=("y", "dx"))
    for k in ("y", "dx"):
        e = rel_err(on[k], off[k])
        say("  on/off", k, "%.2e" % e)
        assert e <= TOL[dt], (k, e)


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
def test_big_tile_table_shape_sampled(orc, dt):
    """The operator-table shape the kernel is chosen for by default (T = 4,
    1024 -> 1024 channels per group element, 32,768 rows): rows spread over
    every row tile and both ends, y and dx against the oracle on those rows
    (the layer acts on each row alone)."""
    from paper_2607_21271_amd import ops
    T, C, N = 4, 1024, 32768
    rs = np.random.RandomState(9400)
    w = synth.round_to(rs.standard_normal((T, C, C)) / np.sqrt(T * C), dt)
    b = synth.round_to(0.1 * rs.standard_normal(C), dt)
    x = synth.round_to(rs.standard_normal((N, C, T)).astype(np.float32), dt)
    dy = synth.round_to(rs.standard_normal((N, C, T)).astype(np.float32), dt)
    wt, bt, xt, dyt = to_dev(w, dt), to_dev(b, dt), to_dev(x, dt), to_dev(dy, dt)
    wspec = ops.weight_spectrum(wt)
    y = ops.forward(xt, wspec, bt, T, C, C)
    dx = ops.backward_input(dyt, wspec, T, C, C)
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([[0, 1, 127, 128, N - 129, N - 1], rs.randint(0, N, 18)]))
    wd, bd = w.astype(np.float64), b.astype(np.float64)
    ry = orc.forward(x[rows].astype(np.float64), wd, bd)
    rdx = orc.backward_input(dy[rows].astype(np.float64), wd)
    idx = torch.from_numpy(rows).cuda()
    ey = rel_err(y[idx].float().cpu().numpy(), ry)
    edx = rel_err(dx[idx].float().cpu().numpy(), rdx)
    say("  table shape", dt, "y %.2e dx %.2e" % (ey, edx))
    assert ey <= TOL[dt] and edx <= TOL[dt], (ey, edx)


WG_CASES = [(4, 32, 128, 128, True), (4, 64, 200, 300, True), (2, 96, 256, 777, True),
            (4, 160, 96, 1000, False), (4, 300, 130, 2000, True), (2, 256, 64, 129, False),
            (4, 384, 256, 2100, True), (4, 16, 40, 33, True)]


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("T,Cin,Cout,N,bias", WG_CASES, ids=["T%d-%dx%d-N%d" % c[:4] for c in WG_CASES])
def test_big_wgrad_matches_oracle(orc, monkeypatch, T, Cin, Cout, N, bias, dt):
    """dw and db of the forced large-tile weight gradient (single split for
    the small row counts, several for the 384 x 256 and 300 x 130 cases)."""
    say("big wgrad", T, Cin, Cout, N, bias, dt)
    monkeypatch.setenv("EQL_WGRAD_KIND", "2")
    inp = synth.draw(T, Cin, Cout, N, bias, 9500 + 13 * T + Cin + Cout).rounded(dt)
    g = run_gpu(inp, dt, want=("dw",))
    ref_dw, ref_db = orc.backward_weight(inp.x, inp.dy, with_bias=bias)
    errs = {"dw": rel_err(g["dw"], ref_dw)}
    if bias:
        errs["db"] = rel_err(g["db"], ref_db)
    say("  ", {k: "%.2e" % v for k, v in errs.items()})
    for k, v in errs.items():
        assert v <= TOL[dt], (k, v)


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
def test_big_whole_backward_default_plan(orc, dt):
    """A layer wide enough for both large-tile kernels by default (1024 ->
    1024 at T = 4; 520 rows keep the fp64 oracle fast): the whole backward
    (eqlinear_backward) and the forward against the oracle."""
    from paper_2607_21271_amd import ops
    T, Cin, Cout, N = 4, 1024, 1024, 520
    inp = synth.draw(T, Cin, Cout, N, True, 9600).rounded(dt)
    x, w, dy, b = to_dev(inp.x, dt), to_dev(inp.w, dt), to_dev(inp.dy, dt), to_dev(inp.b, dt)
    wspec = ops.weight_spectrum(w)
    y = ops.forward(x, wspec, b, T, Cin, Cout)
    dx, dw, db = ops.backward(x, dy, wspec, T, Cin, Cout, with_bias=True)
    torch.cuda.synchronize()
    ref_dw, ref_db = orc.backward_weight(inp.x, inp.dy)
    errs = {"y": rel_err(y.float().cpu().numpy(), orc.forward(inp.x, inp.w, inp.b)),
            "dx": rel_err(dx.float().cpu().numpy(), orc.backward_input(inp.dy, inp.w)),
            "dw": rel_err(dw.float().cpu().numpy(), ref_dw),
            "db": rel_err(db.float().cpu().numpy(), ref_db)}
    say("  whole backward", dt, {k: "%.2e" % v for k, v in errs.items()})
    for k, v in errs.items():
        assert v <= TOL[dt], (k, v)


def test_big_fp32_default_plan_at_2048_sampled(orc):
    """fp32 at T = 4, 2048 -> 2048 channels, 2,000 rows: the default plan
    takes the three-product forward and input gradient (96-channel tiles)
    and the three-product weight gradient (16 x 22 tiles of 128 x 96 in 8 row
    splits, 2,816 workgroups).  Sampled rows of y and dx and sampled dw
    entries against the oracle (db of this kernel: the smaller forced cases)."""
    from paper_2607_21271_amd import ops
    T, C, N = 4, 2048, 2000
    rs = np.random.RandomState(9700)
    w = (rs.standard_normal((T, C, C)) / np.sqrt(T * C)).astype(np.float32)
    b = (0.1 * rs.standard_normal(C)).astype(np.float32)
    x = rs.standard_normal((N, C, T)).astype(np.float32)
    dy = rs.standard_normal((N, C, T)).astype(np.float32)
    xt, wt, bt, dyt = to_dev(x, "f32"), to_dev(w, "f32"), to_dev(b, "f32"), to_dev(dy, "f32")
    wspec = ops.weight_spectrum(wt)
    y = ops.forward(xt, wspec, bt, T, C, C)
    dx, dw, _ = ops.backward(xt, dyt, wspec, T, C, C, with_bias=True)
    torch.cuda.synchronize()
    rows = np.unique(np.concatenate([[0, 127, 128, N - 1], rs.randint(0, N, 12)]))
    wd, bd = w.astype(np.float64), b.astype(np.float64)
    ey = rel_err(y.cpu().numpy()[rows], orc.forward(x[rows].astype(np.float64), wd, bd))
    edx = rel_err(dx.cpu().numpy()[rows], orc.backward_input(dy[rows].astype(np.float64), wd))
    jj, oo, cc = rs.randint(0, T, 64), rs.randint(0, C, 64), rs.randint(0, C, 64)
    ref = orc.backward_weight_entries(x, dy, jj, oo, cc)
    got = dw.cpu().numpy()[jj, oo, cc]
    edw = float(np.max(np.abs(got - ref)) / np.max(np.abs(ref)))
    say("  fp32 2048 default", "y %.2e dx %.2e dw %.2e" % (ey, edx, edw))
    for k, v in (("y", ey), ("dx", edx), ("dw", edw)):
        assert v <= TOL["f32"], (k, v)


def test_big_wgrad_noalloc_falls_back_within_scratch():
    """A wide layer whose large-tile plan needs more workspace than the static
    scratch of the allocation-free entry point (1024 x 1024 at T = 4, 4,096
    rows: spectra of 2 x 32 MiB plus partials): that entry point plans the
    split-row kernels instead, and agrees with the workspace entry point to
    the fp16 bar."""
    from paper_2607_21271_amd import _lib as L
    L.lib()
    T, C, N = 4, 1024, 4096
    need = L.eqlinear_backward_weight_workspace_bytes(N, T, C, C, L.EQL_F16)
    assert need > L.STATIC_SCRATCH_BYTES, need
    rs = np.random.RandomState(9700)
    x = torch.from_numpy(rs.standard_normal((N, C, T)).astype(np.float16)).cuda()
    dy = torch.from_numpy(rs.standard_normal((N, C, T)).astype(np.float16)).cuda()
    stream = torch.cuda.current_stream().cuda_stream
    dw_ws = torch.empty(T, C, C, dtype=torch.float16, device="cuda")
    db_ws = torch.empty(C, dtype=torch.float16, device="cuda")
    ws = torch.empty(need, dtype=torch.uint8, device="cuda")
    st = L.eqlinear_backward_weight(x.data_ptr(), dy.data_ptr(), dw_ws.data_ptr(), db_ws.data_ptr(), ws.data_ptr(),
                                    need, N, T, C, C, L.EQL_F16, stream)
    assert st == L.EQL_OK, L.eqlinear_status_string(st)
    dw_na = torch.empty_like(dw_ws)
    db_na = torch.empty_like(db_ws)
    st = L.eqlinear_backward_weight_noalloc(x.data_ptr(), dy.data_ptr(), dw_na.data_ptr(), db_na.data_ptr(), N, T,
                                            C, C, L.EQL_F16, stream)
    assert st == L.EQL_OK, L.eqlinear_status_string(st)
    torch.cuda.synchronize()
    e_dw = rel_err(dw_na.float().cpu().numpy(), dw_ws.float().cpu().numpy())
    e_db = rel_err(db_na.float().cpu().numpy(), db_ws.float().cpu().numpy())
    say("  noalloc vs workspace", "%.2e %.2e" % (e_dw, e_db))
    assert e_dw <= TOL["f16"] and e_db <= TOL["f16"], (e_dw, e_db)


def _random_shapes(n, seed):
    rs = np.random.RandomState(seed)
    out = []
    for _ in range(n):
        T = int(rs.choice([2, 4]))
        Cin = int(32 * rs.randint(1, 14))          # the contraction of the forward
        Cout = int(rs.randint(1, 301))             # anything (the input gradient takes
        N = int(rs.randint(1, 700))                # the large tiles only at multiples of 32)
        out.append((T, Cin, Cout, N, bool(rs.randint(0, 2))))
    return out


RANDOM = _random_shapes(12, 9800)


@pytest.mark.parametrize("dt", ["f32", "f16", "bf16"])
@pytest.mark.parametrize("T,Cin,Cout,N,bias", RANDOM, ids=["T%d-%dx%d-N%d" % c[:4] for c in RANDOM])
def test_big_tile_random_shapes(orc, monkeypatch, T, Cin, Cout, N, bias, dt):
    """Seeded random shapes with both large-tile paths forced: y, dx, dw and
    db against the oracle."""
    say("big random", T, Cin, Cout, N, bias, dt)
    monkeypatch.setenv("EQL_GEMM_BIG", "1")
    monkeypatch.setenv("EQL_WGRAD_KIND", "2")
    inp = synth.draw(T, Cin, Cout, N, bias, 9900 + T + Cin + Cout + N).rounded(dt)
    g = run_gpu(inp, dt)
    ref_dw, ref_db = orc.backward_weight(inp.x, inp.dy, with_bias=bias)
    errs = {"y": rel_err(g["y"], orc.forward(inp.x, inp.w, inp.b)),
            "dx": rel_err(g["dx"], orc.backward_input(inp.dy, inp.w)),
            "dw": rel_err(g["dw"], ref_dw)}
    if bias:
        errs["db"] = rel_err(g["db"], ref_db)
    say("  ", {k: "%.2e" % v for k, v in errs.items()})
    for k, v in errs.items():
        assert v <= TOL[dt], (k, v)
