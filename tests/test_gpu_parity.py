"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle.

Bar (per output tensor): max|gpu - oracle| / max|oracle| <= 1e-5 for fp32 and
<= 5e-3 for fp16, with the oracle fed the same dtype-rounded inputs.
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


# Reduced row counts: several row tiles plus a ragged tail, oracle in seconds.
REDUCED_N = {"tiny_c4": 256, "vit_s_proj": 1037, "vit_b_mlp_up": 517, "vit_b_mlp_down": 517,
             "swin_s1": 2085, "sweep_T3": 1029, "sweep_T5": 1029, "sweep_T12": 1029,
             "sweep_T16": 1029}
CASES = [(name, dt) for name, l in synth.LAYERS.items() for dt in l.dtypes]


def _check_all(inp, dt, orc, tag):
    g = run_gpu(inp, dt)
    y = orc.forward(inp.x, inp.w, inp.b)
    dx = orc.backward_input(inp.dy, inp.w)
    dw, db = orc.backward_weight(inp.x, inp.dy, with_bias=inp.b is not None)
    errs = {"y": rel_err(g["y"], y), "dx": rel_err(g["dx"], dx), "dw": rel_err(g["dw"], dw)}
    if db is not None:
        errs["db"] = rel_err(g["db"], db)
    say(tag, dt, {k: "%.2e" % v for k, v in errs.items()})
    for k, v in errs.items():
        assert v <= TOL[dt], (tag, dt, k, v)
    return g


@pytest.mark.parametrize("name,dt", CASES, ids=["%s-%s" % c for c in CASES])
def test_layer_reduced_rows(orc, name, dt):
    l = synth.LAYERS[name]
    say("case", name, dt, "N =", REDUCED_N[name])
    inp = synth.draw(l.T, l.Cin, l.Cout, REDUCED_N[name], l.bias, l.seed).rounded(dt)
    _check_all(inp, dt, orc, name)


@pytest.mark.parametrize("name,dt", CASES, ids=["%s-%s" % c for c in CASES])
def test_layer_full_size(orc, name, dt):
    """Full workload size, in the launch configuration the benchmark times: every
    element of y, dx, dw and db against the oracle (per-tensor errors as in
    Sec. 4.3, Table 4)."""
    l = synth.LAYERS[name]
    say("case full", name, dt, "N =", l.N)
    inp = synth.draw_layer(l).rounded(dt)
    _check_all(inp, dt, orc, name + " full")


EDGE = []
for T in range(1, 17):
    EDGE.append((T, 5, 7, 37, True))
    EDGE.append((T, 33, 19, 70, False))
EDGE += [(3, 3, 5, 11, True), (5, 1, 1, 1, True), (7, 2, 9, 16, True), (4, 24, 96, 17, False),
         (8, 96, 384, 1, False), (8, 384, 96, 33, False), (16, 64, 64, 65, True),
         (12, 64, 1, 63, True), (2, 129, 130, 31, True), (6, 40, 200, 50, True)]


@pytest.mark.parametrize("dt", ["f32", "f16"])
@pytest.mark.parametrize("T,Cin,Cout,N,bias", EDGE,
                         ids=["T%d-%dx%d-N%d%s" % (e[0], e[1], e[2], e[3], "-b" if e[4] else "")
                              for e in EDGE])
def test_edge_shapes(orc, T, Cin, Cout, N, bias, dt):
    say("edge", T, Cin, Cout, N, bias, dt)
    inp = synth.draw(T, Cin, Cout, N, bias, 9000 + 97 * T + Cin + 7 * Cout + N).rounded(dt)
    _check_all(inp, dt, orc, "edge T%d %dx%d N%d" % (T, Cin, Cout, N))


@pytest.mark.parametrize("dt", ["f32", "f16"])
def test_zero_rows(dt):
    from paper_2607_21271_amd import ops
    T, Cin, Cout = 8, 16, 24
    w = to_dev(np.random.RandomState(1).standard_normal((T, Cout, Cin)), dt)
    b = to_dev(np.ones(Cout), dt)
    wspec = ops.weight_spectrum(w)
    x = torch.empty(0, Cin, T, dtype=w.dtype, device="cuda")
    y = ops.forward(x, wspec, b, T, Cin, Cout)
    dx = ops.backward_input(torch.empty(0, Cout, T, dtype=w.dtype, device="cuda"), wspec, T, Cin, Cout)
    dw = torch.full((T, Cout, Cin), 7.0, dtype=w.dtype, device="cuda")
    db = torch.full((Cout,), 7.0, dtype=w.dtype, device="cuda")
    ops.backward_weight(x, torch.empty(0, Cout, T, dtype=w.dtype, device="cuda"), T, Cin, Cout,
                        True, dw=dw, db=db)
    torch.cuda.synchronize()
    assert y.shape == (0, Cout, T) and dx.shape == (0, Cin, T)
    assert torch.all(dw == 0) and torch.all(db == 0)


@pytest.mark.parametrize("dt", ["f32", "f16"])
def test_bitwise_determinism(dt):
    l = synth.LAYERS["vit_b_mlp_up"] if dt == "f16" else synth.LAYERS["vit_s_proj"]
    inp = synth.draw_layer(l.with_n(3001)).rounded(dt)
    a = run_gpu(inp, dt)
    b = run_gpu(inp, dt)
    for k in a:
        if a[k] is not None:
            assert np.array_equal(a[k], b[k]), k


@pytest.mark.parametrize("dt", ["f32", "f16"])
def test_guard_bands_untouched(dt):
    """Outputs written into views of larger sentinel-filled buffers leave the slack alone."""
    from paper_2607_21271_amd import ops
    T, Cin, Cout, N = 5, 24, 40, 77
    inp = synth.draw(T, Cin, Cout, N, True, 77).rounded(dt)
    x, w, dy, b = to_dev(inp.x, dt), to_dev(inp.w, dt), to_dev(inp.dy, dt), to_dev(inp.b, dt)
    wspec = ops.weight_spectrum(w)
    SENT, PAD = 12345.0, 64   # PAD elements keep 16-byte alignment of the view

    def guarded(n):
        buf = torch.full((PAD + n + PAD,), SENT, dtype=w.dtype, device="cuda")
        return buf, buf[PAD:PAD + n]

    yb, yv = guarded(N * Cout * T)
    dxb, dxv = guarded(N * Cin * T)
    dwb, dwv = guarded(T * Cout * Cin)
    dbb, dbv = guarded(Cout)
    ops.forward(x, wspec, b, T, Cin, Cout, out=yv.view(N, Cout, T))
    ops.backward_input(dy, wspec, T, Cin, Cout, out=dxv.view(N, Cin, T))
    ops.backward_weight(x, dy, T, Cin, Cout, True, dw=dwv.view(T, Cout, Cin), db=dbv)
    torch.cuda.synchronize()
    for buf in (yb, dxb, dwb, dbb):
        assert torch.all(buf[:PAD] == SENT) and torch.all(buf[-PAD:] == SENT)
        assert not torch.any(buf[PAD:-PAD] == SENT)


@pytest.mark.parametrize("dt", ["f32", "f16"])
def test_roll_equivariance_gpu(dt):
    """f(G x) = G f(x): rolling x along the group axis rolls y (Table 5's test)."""
    from paper_2607_21271_amd import ops
    for T in (4, 8, 5):
        inp = synth.draw(T, 32, 48, 300, True, 31 + T).rounded(dt)
        x, w, b = to_dev(inp.x, dt), to_dev(inp.w, dt), to_dev(inp.b, dt)
        wspec = ops.weight_spectrum(w)
        y = ops.forward(x, wspec, b, T, 32, 48).double()
        for r in range(1, T):
            yr = ops.forward(torch.roll(x, r, dims=2).contiguous(), wspec, b, T, 32, 48).double()
            err = (yr - torch.roll(y, r, dims=2)).abs().max().item() / y.abs().max().item()
            assert err <= TOL[dt], (T, r, err)


def test_nan_propagates():
    from paper_2607_21271_amd import ops
    T, Cin, Cout, N = 4, 8, 8, 40
    inp = synth.draw(T, Cin, Cout, N, True, 5).rounded("f32")
    x, w, b = to_dev(inp.x, "f32"), to_dev(inp.w, "f32"), to_dev(inp.b, "f32")
    x[3, 2, 1] = float("nan")
    y = ops.forward(x, ops.weight_spectrum(w), b, T, Cin, Cout)
    torch.cuda.synchronize()
    assert torch.isnan(y[3]).all()
    assert torch.isfinite(y[:3]).all() and torch.isfinite(y[4:]).all()


def test_error_paths_with_device_pointers():
    from paper_2607_21271_amd import _lib, ops
    T, Cin, Cout, N = 4, 8, 8, 16
    w = torch.randn(T, Cout, Cin, device="cuda")
    wspec = ops.weight_spectrum(w)
    buf = torch.randn(N * Cin * T + 1, device="cuda")
    x_mis = buf[1:].view(N, Cin, T)             # 4-byte offset: misaligned
    with pytest.raises(_lib.EqlError) as e:
        ops.forward(x_mis, wspec, None, T, Cin, Cout)
    assert e.value.status == _lib.EQL_ERR_ALIGNMENT
    x = torch.randn(N, Cin, T, device="cuda")
    with pytest.raises(_lib.EqlError) as e:        # y aliases x
        ops.forward(x, wspec, None, T, Cin, Cout, out=x)
    assert e.value.status == _lib.EQL_ERR_INVALID_ARG


def test_autograd_module_matches_oracle(orc):
    from paper_2607_21271_amd.ops import EQLinear
    T, Cin, Cout, N = 8, 24, 40, 130
    inp = synth.draw(T, Cin, Cout, N, True, 4242).rounded("f32")
    m = EQLinear(T, Cin, Cout, bias=True, device="cuda")
    with torch.no_grad():
        m.weight.copy_(torch.from_numpy(inp.w))
        m.bias.copy_(torch.from_numpy(inp.b))
    x = to_dev(inp.x, "f32").view(2, 65, Cin, T).requires_grad_(True)
    y = m(x)
    y.backward(to_dev(inp.dy, "f32").view(2, 65, Cout, T))
    torch.cuda.synchronize()
    ref_y = orc.forward(inp.x, inp.w, inp.b)
    ref_dx = orc.backward_input(inp.dy, inp.w)
    ref_dw, ref_db = orc.backward_weight(inp.x, inp.dy)
    assert rel_err(y.detach().cpu().numpy().reshape(N, Cout, T), ref_y) <= 1e-5
    assert rel_err(x.grad.cpu().numpy().reshape(N, Cin, T), ref_dx) <= 1e-5
    assert rel_err(m.weight.grad.cpu().numpy(), ref_dw) <= 1e-5
    assert rel_err(m.bias.grad.cpu().numpy(), ref_db) <= 1e-5


# The weight mode is chosen from the shape and the row count; each mode is also
# forced here on small inputs so that both instantiations of a shape stay under
# test (0: streamed weights, 2: every weight block resident in LDS, where the
# blocks fit; elsewhere the plan keeps its own mode).
FORCED = [(3, 64, 64, 1029, True), (4, 24, 96, 2085, False), (4, 96, 24, 700, False),
          (5, 64, 64, 515, True), (8, 48, 48, 613, True), (12, 64, 64, 257, True),
          (7, 40, 72, 130, False), (2, 64, 200, 99, True), (8, 96, 384, 300, False)]


@pytest.mark.gpu
@pytest.mark.parametrize("mode", ["0", "2"])
@pytest.mark.parametrize("dt", ["f32", "f16"])
@pytest.mark.parametrize("T,Cin,Cout,N,bias", FORCED,
                         ids=["T%d-%dx%d-N%d" % f[:4] for f in FORCED])
def test_forced_weight_mode(orc, monkeypatch, T, Cin, Cout, N, bias, dt, mode):
    say("forced mode", mode, T, Cin, Cout, N, dt)
    monkeypatch.setenv("EQL_GEMM_MODE", mode)
    inp = synth.draw(T, Cin, Cout, N, bias, 7000 + 31 * T + Cin + Cout).rounded(dt)
    g = run_gpu(inp, dt, want=("y", "dx"))
    errs = {"y": rel_err(g["y"], orc.forward(inp.x, inp.w, inp.b)),
            "dx": rel_err(g["dx"], orc.backward_input(inp.dy, inp.w))}
    say("  ", {k: "%.2e" % v for k, v in errs.items()})
    for k, v in errs.items():
        assert v <= TOL[dt], (T, Cin, Cout, dt, mode, k, v)


# The weight-gradient reduction reads IPW consecutive partial items per plane
# and splits the row splits over G thread groups, in workgroups of 256 threads
# (up to 64 splits) or 1024 (more); all three are chosen on the host from T,
# the split count and the item count.  Every run length that fits the
# workgroup is forced here, with the bias gradient, across group orders and
# split counts on both sides of 64 (the T = 3, N = 20000 case has 125).
RED_CASES = [(3, 64, 64, 3000, True), (8, 96, 384, 900, True), (16, 64, 64, 1500, True),
             (5, 24, 40, 70, True), (3, 64, 64, 20000, True)]


@pytest.mark.gpu
@pytest.mark.parametrize("ipw", ["4", "8", "16", "32", "64"])
@pytest.mark.parametrize("T,Cin,Cout,N,bias", RED_CASES,
                         ids=["T%d-%dx%d-N%d" % f[:4] for f in RED_CASES])
def test_wgrad_reduce_run_length(orc, monkeypatch, T, Cin, Cout, N, bias, ipw):
    say("reduce run length", ipw, T, Cin, Cout, N)
    monkeypatch.setenv("EQL_RED_IPW", ipw)
    inp = synth.draw(T, Cin, Cout, N, bias, 7700 + 31 * T + Cin + Cout).rounded("f32")
    g = run_gpu(inp, "f32", want=("dw",))
    ref_dw, ref_db = orc.backward_weight(inp.x, inp.dy)
    errs = {"dw": rel_err(g["dw"], ref_dw), "db": rel_err(g["db"], ref_db)}
    say("  ", {k: "%.2e" % v for k, v in errs.items()})
    for k, v in errs.items():
        assert v <= TOL["f32"], (T, Cin, Cout, ipw, k, v)


# The weight spectrum reads 16-byte runs of input channels where the weight
# base and row stride allow it and single elements elsewhere; both paths give
# the same bits.
@pytest.mark.gpu
@pytest.mark.parametrize("dt", ["f32", "f16"])
@pytest.mark.parametrize("T,Cin,Cout", [(8, 96, 384), (3, 64, 64), (16, 40, 24), (5, 7, 33)])
def test_weight_spectrum_unaligned_base(T, Cin, Cout, dt):
    from paper_2607_21271_amd import ops
    say("weight spectrum offset base", T, Cin, Cout, dt)
    tdt = torch.float16 if dt == "f16" else torch.float32
    w = (torch.randn(T, Cout, Cin, generator=torch.Generator().manual_seed(T * 1000 + Cin)) /
         np.sqrt(T * Cin)).to(tdt).cuda()
    buf = torch.empty(w.numel() + 1, dtype=tdt, device="cuda")
    w_off = buf[1:].view(T, Cout, Cin)
    w_off.copy_(w)
    assert w_off.data_ptr() % 16 != 0
    a = ops.weight_spectrum(w)
    b = ops.weight_spectrum(w_off)
    torch.cuda.synchronize()
    assert torch.equal(a.cpu(), b.cpu())


# Layers whose contraction fits in at most three MFMA steps and whose output
# spans several o-chunks run the resident-spectrum mode (the activation
# spectrum of a round stays in registers across o-chunks); covered across
# group orders, both passes (the input gradient of the Cin > Cout cases), odd
# and even o-chunk counts and one to three contraction steps.
RES_CASES = [(8, 96, 384, 300, False), (8, 40, 200, 333, True), (8, 384, 96, 260, True),
             (4, 24, 200, 517, False), (4, 200, 24, 300, True), (3, 64, 400, 1029, True),
             (5, 48, 300, 260, True), (7, 32, 256, 130, False), (6, 64, 200, 200, True),
             (2, 96, 512, 99, True), (1, 96, 1024, 77, True)]


@pytest.mark.gpu
@pytest.mark.parametrize("dt", ["f32", "f16"])
@pytest.mark.parametrize("T,Cin,Cout,N,bias", RES_CASES,
                         ids=["T%d-%dx%d-N%d" % f[:4] for f in RES_CASES])
def test_resident_spectrum_mode(orc, T, Cin, Cout, N, bias, dt):
    say("resident spectrum", T, Cin, Cout, N, dt)
    inp = synth.draw(T, Cin, Cout, N, bias, 7900 + 31 * T + Cin + Cout).rounded(dt)
    g = run_gpu(inp, dt, want=("y", "dx"))
    errs = {"y": rel_err(g["y"], orc.forward(inp.x, inp.w, inp.b)),
            "dx": rel_err(g["dx"], orc.backward_input(inp.dy, inp.w))}
    say("  ", {k: "%.2e" % v for k, v in errs.items()})
    for k, v in errs.items():
        assert v <= TOL[dt], (T, Cin, Cout, dt, k, v)


# fp16 activations and gradients of large magnitude: the packed fp16 forward
# transforms then carry partial sums in the thousands (|x| up to about 2300 at
# T = 8, partial sums up to about 18000, below the fp16 limit of 65504).
@pytest.mark.parametrize("T,Cin,Cout,N", [(8, 96, 384, 300), (4, 24, 96, 700), (16, 64, 64, 129),
                                          (5, 48, 40, 257)])
def test_fp16_large_magnitude(orc, T, Cin, Cout, N):
    say("fp16 large magnitude", T, Cin, Cout, N)
    base = synth.draw(T, Cin, Cout, N, True, 6100 + T)
    big = synth.Inputs(base.x * 512.0, base.w, base.b * 512.0, base.dy * 512.0).rounded("f16")
    g = run_gpu(big, "f16", want=("y", "dx"))
    errs = {"y": rel_err(g["y"], orc.forward(big.x, big.w, big.b)),
            "dx": rel_err(g["dx"], orc.backward_input(big.dy, big.w))}
    # the weight gradient sums N*T products: inputs scaled by 8 each keep dw in fp16 range
    mid = synth.Inputs(base.x * 8.0, base.w, base.b, base.dy * 8.0).rounded("f16")
    gw = run_gpu(mid, "f16", want=("dw",))
    ref_dw, ref_db = orc.backward_weight(mid.x, mid.dy)
    errs["dw"] = rel_err(gw["dw"], ref_dw)
    errs["db"] = rel_err(gw["db"], ref_db)
    say("  ", {k: "%.2e" % v for k, v in errs.items()})
    for k, v in errs.items():
        assert v <= TOL["f16"], (T, Cin, Cout, k, v)


# Two host threads, each on its own stream with its own buffers, call all four
# entry points repeatedly at the same time; every result must equal, bit for
# bit, the single-thread result of the same call.
def test_two_host_threads_bitwise():
    import threading

    from paper_2607_21271_amd import ops
    say("two host threads")
    shapes = [(8, 96, 384, 1000, False, "f16"), (5, 24, 40, 333, True, "f32")]
    jobs = []
    for k, (T, Cin, Cout, N, bias, dt) in enumerate(shapes):
        inp = synth.draw(T, Cin, Cout, N, bias, 8800 + k).rounded(dt)
        jobs.append((inp, dt, run_gpu(inp, dt)))

    def work(inp, dt, stream, out, reps=6):
        with torch.cuda.stream(stream):
            for _ in range(reps):
                out.append(run_gpu(inp, dt))

    outs = [[] for _ in jobs]
    streams = [torch.cuda.Stream() for _ in jobs]
    threads = [threading.Thread(target=work, args=(j[0], j[1], s, o))
               for j, s, o in zip(jobs, streams, outs)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    torch.cuda.synchronize()
    for (inp, dt, ref), got in zip(jobs, outs):
        assert len(got) == 6
        for g in got:
            for key in ref:
                if ref[key] is not None:
                    assert np.array_equal(g[key], ref[key]), (dt, key)


# Both weight-gradient kernels, forced: the staged kernel (EQL_WGRAD_KIND=0)
# and the register-direct one (=1) with each of its channel tiles
# (EQL_WGRAD_TILE=CT,OT blocks of 16 x 16) that fits the group order; ragged
# channel counts, row counts that are not whole chunks, and a row count
# smaller than one chunk per wave.
WG_CASES = [(8, 96, 384, 700, False), (4, 24, 96, 1111, False), (3, 64, 64, 517, True),
            (16, 40, 24, 300, True), (5, 7, 33, 45, True), (12, 64, 64, 257, True),
            (1, 33, 17, 80, True), (8, 48, 48, 13, True)]
WG_MODES = ["staged", "rd:1,1", "rd:1,2", "rd:2,1", "rd:2,2", "rd:2,4", "rd:4,2"]


def _rd_fits(T, ct, ot):
    return 4 * T * (ct * ot + 2 * (ct + ot)) <= 400


@pytest.mark.gpu
@pytest.mark.parametrize("mode", WG_MODES)
@pytest.mark.parametrize("dt", ["f32", "f16"])
@pytest.mark.parametrize("T,Cin,Cout,N,bias", WG_CASES, ids=["T%d-%dx%d-N%d" % f[:4] for f in WG_CASES])
def test_wgrad_kernel_forced(orc, monkeypatch, T, Cin, Cout, N, bias, dt, mode):
    if mode == "staged":
        monkeypatch.setenv("EQL_WGRAD_KIND", "0")
    else:
        ct, ot = (int(v) for v in mode[3:].split(","))
        if not _rd_fits(T, ct, ot):
            pytest.skip("tile does not fit this group order")
        monkeypatch.setenv("EQL_WGRAD_KIND", "1")
        monkeypatch.setenv("EQL_WGRAD_TILE", "%d,%d" % (ct, ot))
    say("weight gradient", mode, T, Cin, Cout, N, dt)
    inp = synth.draw(T, Cin, Cout, N, bias, 7300 + 31 * T + Cin + Cout).rounded(dt)
    g = run_gpu(inp, dt, want=("dw",))
    ref_dw, ref_db = orc.backward_weight(inp.x, inp.dy, with_bias=bias)
    errs = {"dw": rel_err(g["dw"], ref_dw)}
    if bias:
        errs["db"] = rel_err(g["db"], ref_db)
    say("  ", {k: "%.2e" % v for k, v in errs.items()})
    for k, v in errs.items():
        assert v <= TOL[dt], (T, Cin, Cout, dt, mode, k, v)
