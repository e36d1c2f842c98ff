"""The allocation-free weight gradient (eqlinear_backward_weight_noalloc), through
the C ABI, against the workspace entry point eqlinear_backward_weight.

Both run the same kernels with the same plan, so their dw and db must agree
bit for bit; each is also within the fp16 / fp32 bar of the oracle.  Two calls
in a row on one GPU, the second with a smaller problem, check that the shared
static scratch carries nothing from one call into the next.
"""
import numpy as np
import pytest

import synth
from gpu_util import TOL, rel_err, say, to_dev

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _both(L, inp, dt):
    T, Cout, Cin = inp.w.shape
    N = inp.x.shape[0]
    code = L.EQL_F16 if dt == "f16" else L.EQL_F32
    x, dy = to_dev(inp.x, dt), to_dev(inp.dy, dt)
    bias = inp.b is not None
    outs = []
    for noalloc in (False, True):
        dw = torch.full((T, Cout, Cin), 7.0, dtype=x.dtype, device="cuda")
        db = torch.full((Cout,), 7.0, dtype=x.dtype, device="cuda") if bias else None
        dbp = db.data_ptr() if bias else None
        stream = torch.cuda.current_stream().cuda_stream
        if noalloc:
            st = L.eqlinear_backward_weight_noalloc(x.data_ptr(), dy.data_ptr(), dw.data_ptr(), dbp, N,
                                                    T, Cin, Cout, code, stream)
        else:
            need = L.eqlinear_backward_weight_workspace_bytes(N, T, Cin, Cout, code)
            ws = torch.empty(max(need, 1), dtype=torch.uint8, device="cuda")
            st = L.eqlinear_backward_weight(x.data_ptr(), dy.data_ptr(), dw.data_ptr(), dbp,
                                            ws.data_ptr(), need, N, T, Cin, Cout, code, stream)
        assert st == L.EQL_OK, (noalloc, st, L.eqlinear_status_string(st))
        torch.cuda.synchronize()
        outs.append((dw.float().cpu().numpy(), db.float().cpu().numpy() if bias else None))
    return outs


def test_noalloc_matches_workspace_entry_point_twice(orc):
    from paper_2607_21271_amd import _lib as L
    L.lib()
    cases = [("vit_b_mlp_up", "f16", None), ("sweep_T5", "f32", 333)]
    for name, dt, rows in cases:
        l = synth.LAYERS[name]
        n = rows or l.N
        say("no-alloc weight gradient", name, dt, "N =", n)
        inp = synth.draw(l.T, l.Cin, l.Cout, n, l.bias, l.seed).rounded(dt)
        (dw_ws, db_ws), (dw_na, db_na) = _both(L, inp, dt)
        assert np.array_equal(dw_ws, dw_na), name
        if db_ws is not None:
            assert np.array_equal(db_ws, db_na), name
        ref_dw, ref_db = orc.backward_weight(inp.x, inp.dy, with_bias=inp.b is not None)
        assert rel_err(dw_na, ref_dw) <= TOL[dt], name
        if ref_db is not None:
            assert rel_err(db_na, ref_db) <= TOL[dt], name
