"""The drop-in block's host-side structure (paper_2607_21271_amd/blocks.py), on the CPU.

The naive unrolled layer is checked against the fp64 oracle, and the block
built from it is equivariant to rolling the group axis of every token, while
the same block with dense (standard) layers is not, as Sec. 4.3 / Table 5
report for standard layers.  The GPU block with this library's layers is
checked against this one in tests/test_gpu_blocks.py.
"""
import numpy as np
import pytest

torch = pytest.importorskip("torch")

import synth  # noqa: E402


def test_naive_layer_matches_oracle(orc):
    from paper_2607_21271_amd.blocks import NaiveEQLinear
    inp = synth.draw(5, 7, 6, 11, True, 123)
    lay = NaiveEQLinear(5, 7, 6, dtype=torch.float64)
    with torch.no_grad():
        lay.weight.copy_(torch.from_numpy(inp.w))
        lay.bias.copy_(torch.from_numpy(inp.b))
        y = lay(torch.from_numpy(inp.x)).numpy()
    ref = orc.forward(inp.x, inp.w, inp.b)
    assert np.max(np.abs(y - ref)) <= 1e-12 * np.max(np.abs(ref))


@pytest.mark.parametrize("T", [3, 4, 8])
def test_naive_block_equivariant_standard_not(T):
    from paper_2607_21271_amd.blocks import EQViTBlock
    torch.manual_seed(T)
    x = torch.randn(2, 9, 12, T, dtype=torch.float64)
    for lin, expect_equivariant in (("naive", True), ("standard", False)):
        blk = EQViTBlock(T, 12, 3, linear=lin, dtype=torch.float64)
        with torch.no_grad():
            y = blk(x)
            for r in range(1, T):
                err = float((blk(torch.roll(x, r, dims=-1)) - torch.roll(y, r, dims=-1)).abs().max()
                            / y.abs().max())
                if expect_equivariant:
                    assert err <= 1e-12, (lin, T, r, err)
                else:
                    assert err >= 1e-3, (lin, T, r, err)
