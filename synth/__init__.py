"""Seeded synthetic inputs and the workload table for the C_T equivariant linear layer.

This module holds no arithmetic of the method: it only draws Gaussian tensors
from a frozen-stream generator and names the layer shapes.  Both the oracle
side and the GPU side of every test and benchmark take their inputs from here.

Input recipe (stand-ins for EQ-ViT / EQ-Swin activations on ImageNet-100,
which are not available): ``numpy.random.RandomState(seed).standard_normal``
in float64, drawn in the order x (N*Cin*T), w (T*Cout*Cin) scaled by
1/sqrt(T*Cin), b (Cout) scaled by 0.1 when the layer has a bias, dy (N*Cout*T).
The N(0, s) of each workload description is read with s the variance.  Each
tensor is then rounded to the run dtype (round-to-nearest-even; bfloat16 via
float32) and the oracle consumes exactly those rounded values.

Layer shapes follow the paper's EQ-ViT / EQ-Swin configurations (Table 6) and
its operator benchmark rows (Sec. 4.1): 64*197 = 12608 tokens for a ViT batch
of 64 at 224/16 with a class token, 128*56*56 = 401408 tokens for a Swin
stage-1 batch of 128 at 224/4, and 32768 = B*N of the operator benchmark.
"""
from __future__ import annotations

from dataclasses import dataclass, field, replace

import numpy as np

DTYPES = {"f32": np.float32, "f16": np.float16}
# bfloat16 has no numpy type: its values are held in float32 arrays
STORAGE = {"f32": np.float32, "f16": np.float16, "bf16": np.float32}


def _to_bf16(a) -> np.ndarray:
    """float32 array of the bfloat16 numbers nearest to ``a`` (rounded to float32
    first, then to 8 significand bits, round-to-nearest-even on the bit
    pattern).  Finite inputs only."""
    f = np.ascontiguousarray(np.asarray(a, dtype=np.float32))
    bits = f.view(np.uint32).astype(np.uint64)
    bits = (bits + 0x7FFF + ((bits >> 16) & 1)) & 0xFFFF0000
    return bits.astype(np.uint32).view(np.float32).reshape(f.shape)


def round_to(a, dtype: str) -> np.ndarray:
    """``a`` rounded to the values of ``dtype`` (f32, f16 or bf16), in the
    array type that holds them (``STORAGE``)."""
    if dtype == "bf16":
        return _to_bf16(a)
    return np.asarray(a).astype(DTYPES[dtype])


@dataclass(frozen=True)
class Layer:
    name: str
    T: int
    Cin: int
    Cout: int
    N: int
    bias: bool
    seed: int
    dtypes: tuple = ("f32",)
    note: str = ""

    def with_n(self, n: int) -> "Layer":
        return replace(self, N=n)


def _layers():
    out = [
        Layer("tiny_c4", 4, 16, 16, 256, True, 1000, ("f32",),
              "tiny C_4 layer; the oracle finishes in well under a second"),
        Layer("vit_s_proj", 8, 48, 48, 64 * 197, True, 2000, ("f32", "f16"),
              "EQ-ViT-S attention projection, 384-wide embedding at T=8"),
        Layer("vit_b_mlp_up", 8, 96, 384, 64 * 197, False, 3000, ("f16",),
              "EQ-ViT-B MLP up-projection 768 -> 3072 at T=8"),
        Layer("vit_b_mlp_down", 8, 384, 96, 64 * 197, False, 3001, ("f16",),
              "EQ-ViT-B MLP down-projection 3072 -> 768 at T=8"),
        Layer("swin_s1", 4, 24, 96, 128 * 56 * 56, False, 4000, ("f16",),
              "EQ-Swin stage-1 MLP up-projection 96 -> 384 at T=4 (large N, small C)"),
    ]
    for T in (3, 5, 12, 16):
        out.append(Layer(f"sweep_T{T}", T, 64, 64, 32768, True, 5000 + T, ("f32", "f16"),
                         "group-order sweep, odd and non-power-of-two T"))
    return out


LAYERS = {l.name: l for l in _layers()}

# The headline workload: the EQ-ViT-B MLP up-projection, fp16.
HEADLINE = "vit_b_mlp_up"


@dataclass
class Inputs:
    """One draw of the four tensors of a layer, kept in float64 before rounding."""
    x: np.ndarray            # [N, Cin, T]
    w: np.ndarray            # [T, Cout, Cin]
    b: np.ndarray | None     # [Cout] or None
    dy: np.ndarray           # [N, Cout, T]
    extra: dict = field(default_factory=dict)

    def rounded(self, dtype: str) -> "Inputs":
        """The same draw rounded to ``dtype`` (held as ``STORAGE[dtype]``)."""
        r = lambda a: round_to(a, dtype)
        return Inputs(r(self.x), r(self.w), None if self.b is None else r(self.b), r(self.dy))


def draw(T: int, Cin: int, Cout: int, N: int, bias: bool, seed: int) -> Inputs:
    """Draw x, w, b, dy for one layer shape from ``RandomState(seed)``."""
    rs = np.random.RandomState(seed)
    x = rs.standard_normal(N * Cin * T).reshape(N, Cin, T)
    w = (rs.standard_normal(T * Cout * Cin) / np.sqrt(T * Cin)).reshape(T, Cout, Cin)
    b = rs.standard_normal(Cout) * 0.1 if bias else None
    dy = rs.standard_normal(N * Cout * T).reshape(N, Cout, T)
    return Inputs(x, w, b, dy)


def draw_layer(layer: Layer) -> Inputs:
    return draw(layer.T, layer.Cin, layer.Cout, layer.N, layer.bias, layer.seed)
