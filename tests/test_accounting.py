"""Host-side work accounting against the paper's printed counts (CPU only)."""
import os

import numpy as np

from paper_2607_21271_amd import roofline as rf

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _table1():
    rows = {}
    with open(os.path.join(GOLDEN, "table1_c64_counts.txt")) as f:
        for line in f:
            if line.startswith("#") or not line.strip():
                continue
            name, p, g = line.split()
            rows[name] = (float(p), float(g))
    return rows


def test_table1_c64_params_and_flops():
    """Table 1 at c = 64, T = 4, C = D = 256, one sample of 1024 tokens."""
    rows = _table1()
    T, c, N = 4, 64, 1024
    C = D = c * T
    assert round(rf.standard_params(C, D) / 1e6, 3) == rows["standard_linear"][0]
    assert round(rf.eq_params(T, c, c) / 1e6, 3) == rows["naive_eqlinear"][0]
    assert round(rf.eq_params(T, c, c) / 1e6, 3) == rows["flash_eqlinear"][0]
    assert round(rf.standard_linear_flops(N, C, D) / 1e9, 3) == rows["standard_linear"][1]
    assert round(rf.dense_equiv_flops(N, T, c, c) / 1e9, 3) == rows["naive_eqlinear"][1]
    assert round(rf.paper_flash_flops(N, T, c, c) / 1e9, 3) == rows["flash_eqlinear"][1]


def test_p4_products_are_six_sixteenths():
    """Sec. 3.2.2: p4 Step 2 is six real GEMMs, 6/16 of the dense cost."""
    assert rf.real_products(4) == 6
    assert rf.pass_flops(10, 4, 8, 8) / rf.dense_equiv_flops(10, 4, 8, 8) == 6 / 16


def test_bins_cover_T_reals():
    """R + 2K = T: the non-redundant spectrum holds exactly T reals (real-DFT symmetry)."""
    for T in range(1, 17):
        R, K = rf.bins(T)
        assert R + 2 * K == T
        # bins 0..floor(T/2) of numpy's rfft: R of them are real for a real signal
        z = np.fft.rfft(np.random.RandomState(T).standard_normal(T))
        assert len(z) == R + K
        real_bins = [0] + ([T // 2] if T % 2 == 0 else [])
        assert all(abs(z[k].imag) < 1e-12 for k in real_bins)
