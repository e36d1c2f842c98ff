"""GPU parity of the large-tile forward / input-gradient kernel
(csrc/eql_gemm_big.h: 128 x 128 output tiles, 16-bit elements, T in {2, 4})
against the fp64 oracle, through the C ABI.

The host takes this kernel for wide layers only; EQL_GEMM_BIG=1 forces it
wherever the shape allows (contraction channels a multiple of 32), so small
shapes with ragged rows and ragged output-channel tiles cover its tails.  A
pass whose contraction channels are not a multiple of 32 keeps the other
kernel (the input gradient of the Cout = 200 case).  Bar as for the layer:
max|gpu - oracle| / max|oracle| <= 5e-3 (fp16), 4e-2 (bf16).
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


@pytest.mark.parametrize("dt", ["f16", "bf16"])
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


@pytest.mark.parametrize("dt", ["f16", "bf16"])
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


@pytest.mark.parametrize("dt", ["f16", "bf16"])
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
