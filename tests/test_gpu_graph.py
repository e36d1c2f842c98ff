"""The hot path captured in a HIP graph and replayed.

Every launch of the library is a plain kernel launch on the caller's stream
(no memset, no allocation, no host synchronisation), so the four calls of one
step can be recorded in a graph.  Each case records weight spectrum, forward,
input gradient and weight gradient once, then replays the graph several times
with eager work between the replays (outputs cleared by fill kernels, an
unrelated eager launch of the library, synchronisations) and checks that
every replay reproduces the eager results bit for bit (the kernels are
deterministic).
"""
import numpy as np
import pytest

import synth
from gpu_util import say, to_dev

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


# (layer, dtype, rows): a resident-spectrum forward, a ragged odd-T case with
# bias, and an fp32 case with bias
CASES = [("vit_b_mlp_up", "f16", 1500), ("sweep_T3", "f16", 777), ("vit_s_proj", "f32", 1037)]


def _step(ops, x, w, b, dy, bufs, T, Cin, Cout, stream):
    wspec, y, dx, dw, db, ws = bufs
    ops.weight_spectrum(w, out=wspec, stream=stream)
    ops.forward(x, wspec, b, T, Cin, Cout, out=y, stream=stream)
    ops.backward_input(dy, wspec, T, Cin, Cout, out=dx, stream=stream)
    ops.backward_weight(x, dy, T, Cin, Cout, with_bias=b is not None, dw=dw, db=db, workspace=ws,
                        stream=stream)


@pytest.mark.parametrize("name,dt,rows", CASES)
def test_graph_replays_match_eager(name, dt, rows):
    from paper_2607_21271_amd import ops
    say("graph replay", name, dt, rows)
    l = synth.LAYERS[name]
    inp = synth.draw(l.T, l.Cin, l.Cout, rows, l.bias, l.seed).rounded(dt)
    T, Cout, Cin = inp.w.shape
    tdt = {"f32": torch.float32, "f16": torch.float16}[dt]
    x, w, dy = to_dev(inp.x, dt), to_dev(inp.w, dt), to_dev(inp.dy, dt)
    b = to_dev(inp.b, dt) if inp.b is not None else None

    def buffers():
        return (torch.empty(ops._lib.eqlinear_weight_spectrum_bytes(T, Cin, Cout, ops._DT[tdt]),
                            dtype=torch.uint8, device="cuda"),
                torch.empty(rows, Cout, T, dtype=tdt, device="cuda"),
                torch.empty(rows, Cin, T, dtype=tdt, device="cuda"),
                torch.empty(T, Cout, Cin, dtype=tdt, device="cuda"),
                torch.empty(Cout, dtype=tdt, device="cuda") if b is not None else None,
                torch.empty(max(1, ops.workspace_bytes(rows, T, Cin, Cout, tdt)), dtype=torch.uint8,
                            device="cuda"))

    eager = buffers()
    _step(ops, x, w, b, dy, eager, T, Cin, Cout, torch.cuda.current_stream())
    torch.cuda.synchronize()
    ref = [t.clone() for t in eager[1:5] if t is not None]

    gb = buffers()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        _step(ops, x, w, b, dy, gb, T, Cin, Cout, torch.cuda.current_stream())
    other = buffers()
    x2 = torch.flip(x, dims=[0]).contiguous()   # other inputs for the eager work in between
    for rep in range(4):
        for t in gb[1:5]:
            if t is not None:
                t.zero_()
        # unrelated eager work of the same library between the replays
        _step(ops, x2, w, b, dy, other, T, Cin, Cout, torch.cuda.current_stream())
        g.replay()
        torch.cuda.synchronize()
        got = [t for t in gb[1:5] if t is not None]
        for k, (a, r) in enumerate(zip(got, ref)):
            assert torch.equal(a, r), (name, dt, "replay", rep, "output", k)
    say("  4 replays bitwise equal to eager")
