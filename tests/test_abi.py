"""C-ABI checks that need no GPU: the library loads, exports what include/eqlinear.h
declares, and rejects bad arguments before touching the device (CPU only)."""
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "eqlinear.h")

L = pytest.importorskip("paper_2607_21271_amd._lib")


def _header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(eqlinear_\w+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(L.LIB_PATH):
        pytest.fail("libeqlinear.so is not built; run __graft_entry__.build()")
    return L.lib()


def _gpu_visible():
    try:
        import torch
        return torch.cuda.device_count() > 0
    except Exception:
        return False


def test_exports_every_declared_symbol(lib):
    names = _header_functions()
    assert len(names) == 20, names
    for n in names:
        assert hasattr(lib, n), n
        assert n in L.SIGNATURES, n


def test_abi_version_matches_header(lib):
    m = re.search(r"#define EQLINEAR_ABI_VERSION (\d+)", open(HEADER).read())
    assert L.eqlinear_abi_version() == int(m.group(1))


def test_status_strings(lib):
    seen = set()
    for s in range(8):
        t = L.eqlinear_status_string(s)
        assert t and t != "unknown status"
        seen.add(t)
    assert len(seen) == 8
    assert L.eqlinear_status_string(99) == "unknown status"
    assert L.eqlinear_status_string(-1) == "unknown status"


def test_weight_spectrum_bytes(lib):
    # T real planes, two padded layouts (rows to whole output-channel chunks, columns to 32)
    assert L.eqlinear_weight_spectrum_bytes(8, 96, 384, L.EQL_F16) == 8 * (384 * 96 + 96 * 384) * 2
    assert L.eqlinear_weight_spectrum_bytes(4, 16, 16, L.EQL_F32) == 4 * (32 * 32 * 2) * 4
    # bf16 shares every shape and layout of fp16
    assert L.eqlinear_weight_spectrum_bytes(8, 96, 384, L.EQL_BF16) == \
        L.eqlinear_weight_spectrum_bytes(8, 96, 384, L.EQL_F16)
    for bad in [(0, 4, 4, 0), (17, 4, 4, 0), (4, 0, 4, 0), (4, 4, 0, 0), (4, 4, 4, 3), (4, 4, 4, -1),
                (4, 65537, 4, 0)]:
        assert L.eqlinear_weight_spectrum_bytes(*bad) == 0, bad


def test_workspace_bytes(lib):
    assert L.eqlinear_backward_weight_workspace_bytes(0, 8, 96, 384, L.EQL_F16) == 0
    a = L.eqlinear_backward_weight_workspace_bytes(12608, 8, 96, 384, L.EQL_F16)
    assert a > 0 and a % 256 == 0
    assert L.eqlinear_backward_weight_workspace_bytes(-1, 8, 96, 384, L.EQL_F16) == 0
    assert L.eqlinear_backward_weight_workspace_bytes(10, 17, 4, 4, L.EQL_F16) == 0
    assert L.eqlinear_backward_weight_workspace_bytes(12608, 8, 96, 384, L.EQL_BF16) > 0
    assert L.eqlinear_backward_weight_workspace_bytes(12608, 8, 96, 384, 3) == 0


A = 0x10000000  # fake, 16-byte aligned device addresses: never dereferenced on these paths
MB = 1 << 20


def test_forward_argument_checks(lib):
    f = L.eqlinear_forward
    ok = (A, A + 8 * MB, None, A + 16 * MB, 100, 4, 8, 8, L.EQL_F32, None)
    def call(**kw):
        args = list(ok)
        names = ["x", "wspec", "bias", "y", "N", "T", "Cin", "Cout", "dtype", "stream"]
        for k, v in kw.items():
            args[names.index(k)] = v
        return f(*args)
    assert call(T=0) == L.EQL_ERR_INVALID_ARG
    assert call(T=17) == L.EQL_ERR_UNSUPPORTED
    assert call(Cin=0) == L.EQL_ERR_INVALID_ARG
    assert call(Cout=-3) == L.EQL_ERR_INVALID_ARG
    assert call(Cout=70000) == L.EQL_ERR_UNSUPPORTED
    assert call(N=-1) == L.EQL_ERR_INVALID_ARG
    assert call(N=1 << 40) == L.EQL_ERR_UNSUPPORTED
    assert call(dtype=7) == L.EQL_ERR_INVALID_ARG
    assert call(x=None) == L.EQL_ERR_INVALID_ARG
    assert call(y=None) == L.EQL_ERR_INVALID_ARG
    assert call(wspec=None) == L.EQL_ERR_INVALID_ARG
    assert call(x=A + 4) == L.EQL_ERR_ALIGNMENT
    assert call(y=A + 16 * MB + 8) == L.EQL_ERR_ALIGNMENT
    assert call(wspec=A + 8 * MB + 2) == L.EQL_ERR_ALIGNMENT
    assert call(bias=A + 24 * MB + 2) == L.EQL_ERR_ALIGNMENT
    assert call(y=A + 16) == L.EQL_ERR_INVALID_ARG           # y overlaps x
    assert call(bias=A + 32) == L.EQL_ERR_INVALID_ARG        # bias inside x
    assert call(wspec=A + 16 * MB) == L.EQL_ERR_INVALID_ARG  # wspec overlaps y


def test_backward_argument_checks(lib):
    g = L.eqlinear_backward_input
    assert g(A, A + 8 * MB, A + 16 * MB, 10, 0, 4, 4, 0, None) == L.EQL_ERR_INVALID_ARG
    assert g(A, A + 8 * MB, A, 10, 4, 4, 4, 0, None) == L.EQL_ERR_INVALID_ARG
    assert g(A + 8, A + 8 * MB, A + 16 * MB, 10, 4, 4, 4, 0, None) == L.EQL_ERR_ALIGNMENT
    h = L.eqlinear_backward_weight
    need = L.eqlinear_backward_weight_workspace_bytes(1000, 8, 16, 16, L.EQL_F32)
    base = [A, A + 8 * MB, A + 16 * MB, A + 17 * MB, A + 24 * MB, need, 1000, 8, 16, 16, L.EQL_F32, None]
    def call(i, v):
        args = list(base)
        args[i] = v
        return h(*args)
    assert call(5, need - 1) == L.EQL_ERR_WORKSPACE
    assert call(4, None) == L.EQL_ERR_WORKSPACE
    assert call(2, None) == L.EQL_ERR_INVALID_ARG
    assert call(0, None) == L.EQL_ERR_INVALID_ARG
    assert call(2, A + 8 * MB + 4) == L.EQL_ERR_INVALID_ARG   # dw overlaps dy
    assert call(3, A + 2) == L.EQL_ERR_ALIGNMENT
    assert call(4, A + 24 * MB + 4) == L.EQL_ERR_ALIGNMENT
    assert call(7, 17) == L.EQL_ERR_UNSUPPORTED
    w = L.eqlinear_weight_spectrum
    assert w(None, A, 4, 4, 4, 0, None) == L.EQL_ERR_INVALID_ARG
    assert w(A + 2, A + MB, 4, 4, 4, 0, None) == L.EQL_ERR_ALIGNMENT
    assert w(A, A + 64, 4, 4, 4, 0, None) == L.EQL_ERR_INVALID_ARG   # wspec overlaps w


@pytest.mark.skipif(_gpu_visible(), reason="would launch on fake addresses when a GPU is present")
def test_valid_arguments_without_device_report_no_device(lib):
    assert L.eqlinear_forward(A, A + 8 * MB, None, A + 16 * MB, 100, 4, 8, 8, 0, None) == \
        L.EQL_ERR_NO_DEVICE
    assert L.eqlinear_weight_spectrum(A, A + MB, 4, 8, 8, 1, None) == L.EQL_ERR_NO_DEVICE


def test_noalloc_argument_checks(lib):
    """The allocation-free weight gradient checks its arguments like the
    workspace entry point, and refuses a problem whose split partials exceed
    its static device scratch, all before any HIP call."""
    g = L.eqlinear_backward_weight_noalloc
    base = [A, A + 8 * MB, A + 16 * MB, A + 17 * MB, 1000, 8, 16, 16, L.EQL_F32, None]

    def call(i, v):
        args = list(base)
        args[i] = v
        return g(*args)
    assert call(2, None) == L.EQL_ERR_INVALID_ARG
    assert call(0, None) == L.EQL_ERR_INVALID_ARG
    assert call(2, A + 8 * MB + 4) == L.EQL_ERR_INVALID_ARG   # dw overlaps dy
    assert call(3, A + 2) == L.EQL_ERR_ALIGNMENT
    assert call(5, 17) == L.EQL_ERR_UNSUPPORTED
    assert call(8, 5) == L.EQL_ERR_INVALID_ARG
    GB = 1 << 30
    T, C, N = 16, 2048, 1000
    need = L.eqlinear_backward_weight_workspace_bytes(N, T, C, C, L.EQL_F32)
    assert need > L.STATIC_SCRATCH_BYTES
    assert g(A, A + GB, A + 2 * GB, None, N, T, C, C, L.EQL_F32, None) == L.EQL_ERR_SCRATCH
    m = re.search(r"#define EQLINEAR_STATIC_SCRATCH_BYTES \(\(size_t\)(\d+) << (\d+)\)", open(HEADER).read())
    assert int(m.group(1)) << int(m.group(2)) == L.STATIC_SCRATCH_BYTES


def _a256(v):
    return (v + 255) // 256 * 256


def test_large_tile_weight_gradient_plan_and_workspace(lib, monkeypatch):
    """Wide layers with T = 2 or 4 plan the large-tile weight gradient, whose
    workspace holds the fp32 partials of its row splits plus the
    row-contiguous transformed x and dy (T x C rounded up to the channel
    tiles x N rounded up to 64, in the layer's element size); narrower
    layers and other T keep the split-row plans.  fp32 at T = 4 takes
    96-channel o-tiles (three-product bins) where 128-channel tiles alone
    number 256 or more, unless EQL_GAUSS=0; the row splits are as many as
    fill whole rounds of 256 workgroups best.  Host-side queries, no
    device."""
    monkeypatch.delenv("EQL_WGRAD_KIND", raising=False)
    monkeypatch.delenv("EQL_GAUSS", raising=False)
    q = L.eqlinear_backward_weight_workspace_bytes
    T, C, N = 4, 2048, 32768
    NP = N + 64  # 512 blocks of 64 rows, even: one more, for an odd row pitch in 128-byte lines
    # 16 x 16 channel tiles of 128 fill 256 CUs: one split
    spec = T * C * NP * 2
    want = _a256(1 * T * C * C * 4) + _a256(C * 4) + 2 * _a256(spec)
    assert q(N, T, C, C, L.EQL_F16) == want
    assert q(N, T, C, C, L.EQL_BF16) == want
    # fp32: 16 c-tiles x 22 o-tiles of 96 (2112 padded) = 352 tiles; 8 splits
    # make 2816 workgroups, 11 whole rounds
    co = 2112
    want32 = _a256(8 * T * co * C * 4) + _a256(8 * co * 4) + _a256(T * C * NP * 4) + _a256(T * co * NP * 4)
    assert q(N, T, C, C, L.EQL_F32) == want32
    monkeypatch.setenv("EQL_GAUSS", "0")
    assert q(N, T, C, C, L.EQL_F32) == _a256(T * C * C * 4) + _a256(C * 4) + 2 * _a256(T * C * NP * 4)
    monkeypatch.delenv("EQL_GAUSS")
    # 1030 -> 1100 channels at 5,000 rows: both pad to 1152, N to 5,056 (79 blocks)
    Ci, Co, n = 1030, 1100, 5000
    got = q(n, T, Ci, Co, L.EQL_F16)
    assert got >= 2 * _a256(T * 1152 * 5056 * 2)
    # 9 x 9 tiles: 3 splits (243 workgroups, one round), not 4 (324, two)
    assert got == _a256(3 * T * 1152 * 1152 * 4) + _a256(3 * 1152 * 4) + 2 * _a256(T * 1152 * 5056 * 2)
    # below the thresholds (fp16 and fp32 768, bf16 512), T = 8: no spectra
    for args in ((N, T, 512, 512, L.EQL_F16), (N, T, 256, 256, L.EQL_BF16), (N, T, 512, 512, L.EQL_F32),
                 (N, 8, C, C, L.EQL_F16)):
        assert q(*args) < args[0] * args[1] * (args[2] + args[3]) * 2, args
    assert q(N, T, 512, 512, L.EQL_BF16) > N * T * 1024 * 2
    # fp32 at 1024: 8 x 8 tiles of 128 (four products), 4 splits
    assert q(N, T, 1024, 1024, L.EQL_F32) == (_a256(4 * T * 1024 * 1024 * 4) + _a256(4 * 1024 * 4)
                                              + 2 * _a256(T * 1024 * NP * 4))
    # forced on a small layer
    small = q(1000, 2, 64, 96, L.EQL_F16)
    monkeypatch.setenv("EQL_WGRAD_KIND", "2")
    assert q(1000, 2, 64, 96, L.EQL_F16) >= _a256(2 * 128 * 1024 * 2) * 2
    assert q(1000, 2, 64, 96, L.EQL_F32) >= _a256(2 * 128 * 1024 * 4) * 2
    monkeypatch.delenv("EQL_WGRAD_KIND")
    assert q(1000, 2, 64, 96, L.EQL_F16) == small


def test_noalloc_plans_within_static_scratch(lib):
    """The allocation-free entry point takes the split-row plan where the
    large-tile workspace exceeds its scratch (so it does not refuse a wide
    layer that the split-row kernels can handle): with no device it reaches
    the device check (EQL_ERR_NO_DEVICE), not EQL_ERR_SCRATCH."""
    T, C, N = 4, 1024, 4096
    assert L.eqlinear_backward_weight_workspace_bytes(N, T, C, C, L.EQL_F16) > L.STATIC_SCRATCH_BYTES
    GB = 1 << 30
    st = L.eqlinear_backward_weight_noalloc(A, A + GB, A + 2 * GB, None, N, T, C, C, L.EQL_F16, None)
    if _gpu_visible():
        pytest.skip("a device is visible: the call would launch")
    assert st == L.EQL_ERR_NO_DEVICE, L.eqlinear_status_string(st)


def test_whole_backward_plan_and_workspace(lib):
    """eqlinear_backward fuses large row counts against a small tile (Swin
    stage 1) and not the EQ-ViT-B MLP (96 x 384 x 8 does not fit one
    workgroup); its workspace query follows the chosen path."""
    assert L.eqlinear_backward_is_fused(401408, 4, 24, 96, L.EQL_F16) == 1
    assert L.eqlinear_backward_is_fused(401408, 4, 24, 96, L.EQL_F32) == 0   # fp16 only
    assert L.eqlinear_backward_is_fused(12608, 8, 96, 384, L.EQL_F16) == 0
    assert L.eqlinear_backward_is_fused(12608, 8, 48, 48, L.EQL_F16) == 0   # no variant at T = 8 holds it
    assert L.eqlinear_backward_is_fused(32768, 3, 64, 64, L.EQL_F16) == 1
    assert L.eqlinear_backward_is_fused(32768, 3, 64, 64, L.EQL_F32) == 0
    assert L.eqlinear_backward_is_fused(4096, 3, 64, 64, L.EQL_F16) == 0    # partials would dominate
    assert L.eqlinear_backward_is_fused(10 ** 7, 16, 16, 16, L.EQL_F32) == 0  # no variant built for T = 16
    assert L.eqlinear_backward_is_fused(0, 4, 24, 96, L.EQL_F16) == 0
    assert L.eqlinear_backward_is_fused(100, 17, 4, 4, L.EQL_F16) == 0
    assert L.eqlinear_backward_workspace_bytes(12608, 8, 96, 384, L.EQL_F16) == \
        L.eqlinear_backward_weight_workspace_bytes(12608, 8, 96, 384, L.EQL_F16)
    # fused: 256 splits of a 32 x 128 tile, 4 planes of fp32, plus the bias partials
    assert L.eqlinear_backward_workspace_bytes(401408, 4, 24, 96, L.EQL_F16) == \
        256 * 4 * 32 * 128 * 4 + 256 * 128 * 4
    assert L.eqlinear_backward_workspace_bytes(0, 4, 24, 96, L.EQL_F16) == 0
    # bf16 always runs the two passes
    assert L.eqlinear_backward_is_fused(401408, 4, 24, 96, L.EQL_BF16) == 0
    assert L.eqlinear_backward_workspace_bytes(401408, 4, 24, 96, L.EQL_BF16) == \
        L.eqlinear_backward_weight_workspace_bytes(401408, 4, 24, 96, L.EQL_BF16)


def test_whole_backward_forced_plan(lib, monkeypatch):
    monkeypatch.setenv("EQL_BWD_FUSED", "1")
    assert L.eqlinear_backward_is_fused(100, 4, 24, 96, L.EQL_F16) == 1
    assert L.eqlinear_backward_is_fused(100, 4, 24, 96, L.EQL_F32) == 1
    assert L.eqlinear_backward_is_fused(100, 11, 13, 21, L.EQL_F32) == 1
    assert L.eqlinear_backward_is_fused(100, 11, 13, 21, L.EQL_F16) == 0   # no fp16 variant at T = 11
    assert L.eqlinear_backward_is_fused(100, 8, 96, 384, L.EQL_F16) == 0     # no variant holds it
    assert L.eqlinear_backward_is_fused(100, 4, 24, 96, L.EQL_BF16) == 0     # never for bf16
    monkeypatch.setenv("EQL_BWD_FUSED", "0")
    assert L.eqlinear_backward_is_fused(401408, 4, 24, 96, L.EQL_F16) == 0


def test_whole_backward_argument_checks(lib):
    f = L.eqlinear_backward
    N, T, Cin, Cout = 1000, 4, 24, 96
    need = L.eqlinear_backward_workspace_bytes(N, T, Cin, Cout, L.EQL_F32)
    base = [A, A + 8 * MB, A + 16 * MB, A + 24 * MB, A + 32 * MB, A + 33 * MB, A + 40 * MB, need,
            N, T, Cin, Cout, L.EQL_F32, None]
    names = ["x", "dy", "wspec", "dx", "dw", "db", "ws", "wsb", "N", "T", "Cin", "Cout", "dtype",
             "stream"]

    def call(**kw):
        args = list(base)
        for k, v in kw.items():
            args[names.index(k)] = v
        return f(*args)
    assert call(T=0) == L.EQL_ERR_INVALID_ARG
    assert call(T=17) == L.EQL_ERR_UNSUPPORTED
    assert call(dtype=3) == L.EQL_ERR_INVALID_ARG
    for k in ("x", "dy", "wspec", "dx", "dw"):
        assert call(**{k: None}) == L.EQL_ERR_INVALID_ARG, k
    assert call(db=None) != L.EQL_ERR_INVALID_ARG
    assert call(x=A + 4) == L.EQL_ERR_ALIGNMENT
    assert call(dx=A + 24 * MB + 8) == L.EQL_ERR_ALIGNMENT
    assert call(wspec=A + 16 * MB + 2) == L.EQL_ERR_ALIGNMENT
    assert call(dw=A + 32 * MB + 2) == L.EQL_ERR_ALIGNMENT
    assert call(ws=A + 40 * MB + 4) == L.EQL_ERR_ALIGNMENT
    assert call(wsb=need - 1) == L.EQL_ERR_WORKSPACE
    assert call(ws=None) == L.EQL_ERR_WORKSPACE
    assert call(dx=A + 16) == L.EQL_ERR_INVALID_ARG           # dx overlaps x
    assert call(dw=A + 8 * MB) == L.EQL_ERR_INVALID_ARG       # dw overlaps dy
    assert call(ws=A + 24 * MB) == L.EQL_ERR_INVALID_ARG      # workspace overlaps dx
    # N = 0: row tensors may be NULL, no workspace needed
    r = call(N=0, x=None, dy=None, dx=None, ws=None, wsb=0)
    assert r in (L.EQL_OK, L.EQL_ERR_NO_DEVICE)


def test_dihedral_argument_checks(lib):
    """The dihedral weight expansion and gradient fold check shapes, pairing of
    the bias pointers, alignment and overlap before any HIP call."""
    T, Cin, Cout = 4, 6, 10
    for f, nin, nout in ((L.eqlinear_dihedral_expand, 2 * T * Cin * Cout, 4 * T * Cin * Cout),
                         (L.eqlinear_dihedral_fold, 4 * T * Cin * Cout, 2 * T * Cin * Cout)):
        base = [A, A + 8 * MB, A + 16 * MB, A + 24 * MB, T, Cin, Cout, L.EQL_F32, None]

        def call(i, v, f=f):
            args = list(base)
            args[i] = v
            return f(*args)
        assert call(4, 0) == L.EQL_ERR_INVALID_ARG
        assert call(4, 17) == L.EQL_ERR_UNSUPPORTED
        assert call(5, 0) == L.EQL_ERR_INVALID_ARG
        assert call(6, -1) == L.EQL_ERR_INVALID_ARG
        assert call(5, 40000) == L.EQL_ERR_UNSUPPORTED       # 2 Cin over 65536
        assert call(5, 2 ** 30 + 1) == L.EQL_ERR_UNSUPPORTED  # no overflow of 2 Cin
        assert call(7, 9) == L.EQL_ERR_INVALID_ARG
        assert call(0, None) == L.EQL_ERR_INVALID_ARG
        assert call(2, None) == L.EQL_ERR_INVALID_ARG
        assert call(1, None) == L.EQL_ERR_INVALID_ARG        # one bias pointer without the other
        assert call(3, None) == L.EQL_ERR_INVALID_ARG
        assert call(0, A + 2) == L.EQL_ERR_ALIGNMENT
        assert call(2, A + 4) == L.EQL_ERR_INVALID_ARG       # output overlaps input
        assert call(2, A + nin * 4 - 4) == L.EQL_ERR_INVALID_ARG
        assert f(A, None, A + 16 * MB, None, T, Cin, Cout, L.EQL_F32, None) in (L.EQL_OK, L.EQL_ERR_NO_DEVICE) \
            if not _gpu_visible() else True
        assert nout > 0


def test_gconv_argument_checks(lib):
    """The group-convolution gather, scatter and weight permutations check the
    group order, kernel size, extents, alignment and overlap before any HIP
    call."""
    g, sc = L.eqlinear_gconv_gather, L.eqlinear_gconv_scatter
    pk, up = L.eqlinear_gconv_pack_weight, L.eqlinear_gconv_unpack_weight
    B, H, W, T, Cin, Cout, k = 2, 8, 8, 4, 6, 10, 3
    for f in (g, sc):
        base = [A, A + 64 * MB, B, H, W, T, Cin, k, L.EQL_F32, None]

        def call(i, v, f=f):
            args = list(base)
            args[i] = v
            return f(*args)
        assert call(5, 3) == L.EQL_ERR_UNSUPPORTED          # T not in {1, 2, 4}
        assert call(7, 4) == L.EQL_ERR_UNSUPPORTED          # even kernel
        assert call(7, 9) == L.EQL_ERR_UNSUPPORTED          # kernel above 7
        assert call(7, 0) == L.EQL_ERR_INVALID_ARG
        assert call(6, 0) == L.EQL_ERR_INVALID_ARG
        assert call(6, 8000) == L.EQL_ERR_UNSUPPORTED       # k*k*Cin over 65536
        assert call(2, -1) == L.EQL_ERR_INVALID_ARG
        assert call(8, 5) == L.EQL_ERR_INVALID_ARG
        assert call(0, None) == L.EQL_ERR_INVALID_ARG
        assert call(1, None) == L.EQL_ERR_INVALID_ARG
        assert call(0, A + 2) == L.EQL_ERR_ALIGNMENT
        assert call(1, A + 64) == L.EQL_ERR_INVALID_ARG     # output overlaps input
        if not _gpu_visible():
            assert call(2, 0) in (L.EQL_OK, L.EQL_ERR_NO_DEVICE)   # empty image: no-op
    # the forward with the implicit patch gather
    fw = L.eqlinear_gconv_forward
    base = [A, A + 64 * MB, None, A + 128 * MB, B, H, W, T, 8, Cout, k, L.EQL_F32, None]

    def callf(i, v):
        args = list(base)
        args[i] = v
        return fw(*args)
    assert callf(7, 3) == L.EQL_ERR_UNSUPPORTED             # T not in {1, 2, 4}
    assert callf(8, 6) == L.EQL_ERR_UNSUPPORTED             # Cin not a multiple of 4
    assert callf(10, 4) == L.EQL_ERR_UNSUPPORTED            # even kernel
    assert callf(8, 0) == L.EQL_ERR_INVALID_ARG
    assert callf(1, None) == L.EQL_ERR_INVALID_ARG          # no spectrum
    assert callf(0, None) == L.EQL_ERR_INVALID_ARG
    assert callf(3, None) == L.EQL_ERR_INVALID_ARG
    assert callf(0, A + 4) == L.EQL_ERR_ALIGNMENT
    assert callf(3, A + 16) == L.EQL_ERR_INVALID_ARG        # output overlaps the features
    assert callf(2, A + 64 * MB) == L.EQL_ERR_INVALID_ARG   # bias overlaps the spectrum
    assert callf(11, 7) == L.EQL_ERR_INVALID_ARG
    if not _gpu_visible():
        assert callf(4, 0) in (L.EQL_OK, L.EQL_ERR_NO_DEVICE)
    for f in (pk, up, L.eqlinear_gconv_pack_weight_adjoint):
        base = [A, A + 64 * MB, T, Cin, Cout, k, L.EQL_F16, None]

        def call(i, v, f=f):
            args = list(base)
            args[i] = v
            return f(*args)
        assert call(2, 8) == L.EQL_ERR_UNSUPPORTED
        assert call(5, 2) == L.EQL_ERR_UNSUPPORTED
        assert call(4, 0) == L.EQL_ERR_INVALID_ARG
        assert call(0, None) == L.EQL_ERR_INVALID_ARG
        assert call(1, A + 2) == L.EQL_ERR_INVALID_ARG      # overlap
        assert call(0, A + 1) == L.EQL_ERR_ALIGNMENT
