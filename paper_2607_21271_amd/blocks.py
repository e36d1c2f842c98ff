"""Equivariant ViT encoder block with the C_T linear layers as drop-in modules
(Sec. 4.2: every linear layer of EQ-ViT replaced, the rest unchanged).

Tokens carry features [C, T]: C channels per group element and the group axis
T, so a batch is x [B, L, C, T].  The block is

    x = x + proj(attention(qkv(norm1(x))))
    x = x + fc2(gelu(fc1(norm2(x))))

with qkv: C -> 3C, proj: C -> C, fc1: C -> 4C, fc2: 4C -> C all equivariant
linear layers over C_T.  The other parts commute with the group action
(rolling the T axis of every token): the layer norm normalises over (C, T)
with one affine weight and bias per channel, shared over T; attention scores
are dot products over (channels of a head, T); GELU is pointwise.  So the
block is exactly equivariant.

``linear`` selects how the four linear layers run:
  "flash"    this library's layer (EQLinear: rDFT, per-bin MFMA products, irDFT);
  "naive"    the same equivariant weights unrolled into the dense
             [C'T, CT] matrix W[o*T+t, c*T+s] = w[(t-s) mod T, o, c] and
             applied with F.linear (the paper's Naive EQ-Linear);
  "standard" an ordinary dense nn.Linear of the same total widths (C*T -> C'*T),
             not equivariant (the paper's standard ViT baseline).
Weights are random (no trained checkpoint is used); the block serves latency
measurement and equivariance checks.
"""
from __future__ import annotations

import torch
import torch.nn.functional as F

from .ops import EQLinear


class NaiveEQLinear(torch.nn.Module):
    """The equivariant layer through its dense unrolled weight and F.linear."""

    def __init__(self, T: int, Cin: int, Cout: int, bias: bool = True, device=None, dtype=None):
        super().__init__()
        self.T, self.Cin, self.Cout = T, Cin, Cout
        kw = {"device": device, "dtype": dtype}
        self.weight = torch.nn.Parameter(torch.randn(T, Cout, Cin, **kw) / (T * Cin) ** 0.5)
        self.bias = torch.nn.Parameter(torch.zeros(Cout, **kw)) if bias else None
        t = torch.arange(T, device=device)
        self.register_buffer("lag", (t[:, None] - t[None, :]) % T, persistent=False)

    def dense_weight(self):
        T, Cin, Cout = self.T, self.Cin, self.Cout
        return self.weight[self.lag].permute(2, 0, 3, 1).reshape(Cout * T, Cin * T)

    def forward(self, x):
        lead = x.shape[:-2]
        b = None if self.bias is None else self.bias.repeat_interleave(self.T)
        y = F.linear(x.reshape(-1, self.Cin * self.T), self.dense_weight(), b)
        return y.view(*lead, self.Cout, self.T)


class StandardLinear(torch.nn.Module):
    """A dense (not equivariant) linear layer over the flattened [C, T] features."""

    def __init__(self, T: int, Cin: int, Cout: int, bias: bool = True, device=None, dtype=None):
        super().__init__()
        self.T, self.Cin, self.Cout = T, Cin, Cout
        self.lin = torch.nn.Linear(Cin * T, Cout * T, bias=bias, device=device, dtype=dtype)

    def forward(self, x):
        lead = x.shape[:-2]
        return self.lin(x.reshape(-1, self.Cin * self.T)).view(*lead, self.Cout, self.T)


LINEARS = {"flash": EQLinear, "naive": NaiveEQLinear, "standard": StandardLinear}


def _wide(t):
    """fp16 (and bf16) widened to fp32 for reductions; fp32 and fp64 kept."""
    return t.float() if t.dtype in (torch.float16, torch.bfloat16) else t


class GroupLayerNorm(torch.nn.Module):
    """Layer norm over (C, T) with a per-channel affine map shared over T."""

    def __init__(self, C: int, device=None, dtype=None, eps: float = 1e-6):
        super().__init__()
        self.eps = eps
        self.weight = torch.nn.Parameter(torch.ones(C, device=device, dtype=dtype))
        self.bias = torch.nn.Parameter(torch.zeros(C, device=device, dtype=dtype))

    def forward(self, x):
        xf = _wide(x)
        mu = xf.mean(dim=(-2, -1), keepdim=True)
        var = (xf - mu).pow(2).mean(dim=(-2, -1), keepdim=True)
        y = (xf - mu) * torch.rsqrt(var + self.eps)
        y = y * _wide(self.weight)[:, None] + _wide(self.bias)[:, None]
        return y.to(x.dtype)


class EQViTBlock(torch.nn.Module):
    def __init__(self, T: int, C: int, heads: int, mlp_ratio: int = 4, linear: str = "flash",
                 device=None, dtype=None):
        super().__init__()
        assert C % heads == 0
        self.T, self.C, self.heads = T, C, heads
        L = LINEARS[linear]
        kw = {"device": device, "dtype": dtype}
        self.norm1 = GroupLayerNorm(C, **kw)
        self.qkv = L(T, C, 3 * C, **kw)
        self.proj = L(T, C, C, **kw)
        self.norm2 = GroupLayerNorm(C, **kw)
        self.fc1 = L(T, C, mlp_ratio * C, **kw)
        self.fc2 = L(T, mlp_ratio * C, C, **kw)

    def linears(self):
        return [self.qkv, self.proj, self.fc1, self.fc2]

    def attention(self, h):
        B, Lt, _, T = h.shape
        H, dh = self.heads, self.C // self.heads
        qkv = h.view(B, Lt, 3, H, dh * T).permute(2, 0, 3, 1, 4)   # [3, B, H, L, dh*T]
        q, k, v = (qkv[i].contiguous() for i in range(3))
        scores = torch.matmul(q, k.transpose(-1, -2).contiguous()) * (dh * T) ** -0.5
        a = torch.softmax(_wide(scores), dim=-1).to(h.dtype)
        o = torch.matmul(a, v)                                      # [B, H, L, dh*T]
        return o.permute(0, 2, 1, 3).reshape(B, Lt, self.C, T)

    def forward(self, x):
        x = x + self.proj(self.attention(self.qkv(self.norm1(x))))
        x = x + self.fc2(F.gelu(self.fc1(self.norm2(x))))
        return x

    def copy_weights_from(self, other: "EQViTBlock"):
        """Take the equivariant weights of another block (flash <-> naive)."""
        with torch.no_grad():
            for a, b in zip(self.linears(), other.linears()):
                a.weight.copy_(b.weight)
                if a.bias is not None:
                    a.bias.copy_(b.bias)
            for a, b in ((self.norm1, other.norm1), (self.norm2, other.norm2)):
                a.weight.copy_(b.weight)
                a.bias.copy_(b.bias)
