"""Argument checks of the torch front-end (paper_2607_21271_amd/ops.py), on the CPU.

The C ABI receives raw addresses only, so dtype mismatches, wrong output
shapes, non-contiguous outputs and spectra of the wrong size must be refused
in the wrapper before any launch.  Every case here fails in a check that runs
before the device check, so CPU tensors suffice; a call whose arguments are
all consistent fails only because the tensors are not on the GPU.
"""
import pytest

torch = pytest.importorskip("torch")

from paper_2607_21271_amd import ops  # noqa: E402

T, CIN, COUT, N = 4, 8, 12, 5


def spec(dtype=torch.float16):
    return torch.empty(ops.spectrum_bytes(T, CIN, COUT, dtype), dtype=torch.uint8)


def test_consistent_forward_reaches_the_device_check():
    x = torch.zeros(N, CIN, T, dtype=torch.float16)
    with pytest.raises(ValueError, match="GPU"):
        ops.forward(x, spec(), None, T, CIN, COUT)


def test_forward_refuses_spectrum_of_other_dtype():
    x = torch.zeros(N, CIN, T, dtype=torch.float16)
    with pytest.raises(ValueError, match="weight spectrum"):
        ops.forward(x, spec(torch.float32), None, T, CIN, COUT)


def test_forward_refuses_short_or_long_spectrum():
    x = torch.zeros(N, CIN, T, dtype=torch.float32)
    s = spec(torch.float32)
    for bad in (s[:-16], torch.cat([s, s[:16]])):
        with pytest.raises(ValueError, match="weight spectrum"):
            ops.forward(x, bad, None, T, CIN, COUT)


def test_forward_refuses_non_byte_spectrum():
    x = torch.zeros(N, CIN, T, dtype=torch.float32)
    with pytest.raises(TypeError, match="uint8"):
        ops.forward(x, spec(torch.float32).float(), None, T, CIN, COUT)


def test_forward_refuses_bias_dtype_and_shape():
    x = torch.zeros(N, CIN, T, dtype=torch.float16)
    with pytest.raises(TypeError, match="bias"):
        ops.forward(x, spec(), torch.zeros(COUT, dtype=torch.float32), T, CIN, COUT)
    with pytest.raises(ValueError, match="bias"):
        ops.forward(x, spec(), torch.zeros(COUT + 1, dtype=torch.float16), T, CIN, COUT)


def test_forward_refuses_bad_out():
    x = torch.zeros(N, CIN, T, dtype=torch.float16)
    with pytest.raises(ValueError, match="shape"):
        ops.forward(x, spec(), None, T, CIN, COUT, out=torch.empty(N - 1, COUT, T, dtype=torch.float16))
    with pytest.raises(TypeError, match="dtype"):
        ops.forward(x, spec(), None, T, CIN, COUT, out=torch.empty(N, COUT, T, dtype=torch.float32))
    nc = torch.empty(N, T, COUT, dtype=torch.float16).transpose(1, 2)
    with pytest.raises(ValueError, match="contiguous"):
        ops.forward(x, spec(), None, T, CIN, COUT, out=nc)


def test_forward_refuses_wrong_activation_shape_and_dtype():
    with pytest.raises(ValueError, match="x must be"):
        ops.forward(torch.zeros(N, CIN + 1, T, dtype=torch.float16), spec(), None, T, CIN, COUT)
    with pytest.raises(TypeError, match="float32, float16 and bfloat16"):
        ops.forward(torch.zeros(N, CIN, T, dtype=torch.float64), spec(), None, T, CIN, COUT)


def test_backward_input_checks():
    dy = torch.zeros(N, COUT, T, dtype=torch.float16)
    with pytest.raises(ValueError, match="weight spectrum"):
        ops.backward_input(dy, spec(torch.float32), T, CIN, COUT)
    with pytest.raises(ValueError, match="shape"):
        ops.backward_input(dy, spec(), T, CIN, COUT, out=torch.empty(N, COUT, T, dtype=torch.float16))
    with pytest.raises(ValueError, match="GPU"):
        ops.backward_input(dy, spec(), T, CIN, COUT)


def test_backward_weight_checks():
    x = torch.zeros(N, CIN, T, dtype=torch.float16)
    dy = torch.zeros(N, COUT, T, dtype=torch.float16)
    with pytest.raises(TypeError, match="dy"):
        ops.backward_weight(x, dy.float(), T, CIN, COUT)
    with pytest.raises(ValueError, match="rows"):
        ops.backward_weight(x, dy[:-1], T, CIN, COUT)
    with pytest.raises(ValueError, match="dw"):
        ops.backward_weight(x, dy, T, CIN, COUT, dw=torch.empty(T, CIN, COUT, dtype=torch.float16))
    with pytest.raises(TypeError, match="db"):
        ops.backward_weight(x, dy, T, CIN, COUT, db=torch.empty(COUT, dtype=torch.float32))
    need = ops.workspace_bytes(N, T, CIN, COUT, torch.float16)
    assert need > 0
    with pytest.raises(ValueError, match="workspace"):
        ops.backward_weight(x, dy, T, CIN, COUT, workspace=torch.empty(need - 1, dtype=torch.uint8))
    with pytest.raises(ValueError, match="GPU"):
        ops.backward_weight(x, dy, T, CIN, COUT, workspace=torch.empty(need, dtype=torch.uint8))


def test_whole_backward_checks():
    x = torch.zeros(N, CIN, T, dtype=torch.float16)
    dy = torch.zeros(N, COUT, T, dtype=torch.float16)
    with pytest.raises(TypeError, match="dy"):
        ops.backward(x, dy.float(), spec(), T, CIN, COUT)
    with pytest.raises(ValueError, match="rows"):
        ops.backward(x, dy[:-1], spec(), T, CIN, COUT)
    with pytest.raises(ValueError, match="weight spectrum"):
        ops.backward(x, dy, spec(torch.float32), T, CIN, COUT)
    with pytest.raises(ValueError, match="dx"):
        ops.backward(x, dy, spec(), T, CIN, COUT, dx=torch.empty(N, COUT, T, dtype=torch.float16))
    with pytest.raises(ValueError, match="dw"):
        ops.backward(x, dy, spec(), T, CIN, COUT, dw=torch.empty(T, CIN, COUT, dtype=torch.float16))
    with pytest.raises(TypeError, match="db"):
        ops.backward(x, dy, spec(), T, CIN, COUT, db=torch.empty(COUT, dtype=torch.float32))
    need = ops.backward_workspace_bytes(N, T, CIN, COUT, torch.float16)
    assert need > 0
    with pytest.raises(ValueError, match="workspace"):
        ops.backward(x, dy, spec(), T, CIN, COUT, workspace=torch.empty(need - 1, dtype=torch.uint8))
    with pytest.raises(ValueError, match="GPU"):
        ops.backward(x, dy, spec(), T, CIN, COUT)


def test_autograd_function_refuses_mixed_dtypes():
    x = torch.zeros(N, CIN, T, dtype=torch.float16)
    w = torch.zeros(T, COUT, CIN, dtype=torch.float32)
    with pytest.raises(TypeError, match="w has dtype"):
        ops.EQLinearFunction.apply(x, w, None)


def test_spectrum_cache_is_keyed_on_the_weight_version(monkeypatch):
    """The autograd path recomputes the weight spectrum after an in-place update
    of the weight and reuses it otherwise (CPU: the spectrum call is stubbed)."""
    calls = []
    monkeypatch.setattr(ops, "weight_spectrum", lambda w: calls.append(w._version) or object())
    monkeypatch.setattr(ops.torch.cuda, "current_stream", lambda dev=None: type("S", (), {"cuda_stream": 0})())
    w = torch.zeros(T, COUT, CIN)
    a = ops.cached_weight_spectrum(w)
    assert ops.cached_weight_spectrum(w) is a and len(calls) == 1
    w.add_(1.0)
    b = ops.cached_weight_spectrum(w)
    assert b is not a and len(calls) == 2
    w2 = torch.zeros(T, COUT, CIN)
    ops.cached_weight_spectrum(w2)
    assert len(calls) == 3
    n = len(ops._SPEC_CACHE)
    del w2
    assert len(ops._SPEC_CACHE) == n - 1
