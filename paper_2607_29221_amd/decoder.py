"""Secure forward pass of a decoder stack (Section 5.1): every linear layer is
one Pi_Sec-Linear call, every non-linear layer is evaluated by the trusted
client in floating point.

The block is a LLaMA-style pre-norm decoder layer: RMSNorm (gain 1,
eps 1e-5), fused q|k|v projection, causal grouped-query attention (no
rotary embedding), output projection and residual, RMSNorm, fused gate|up
projection, SwiGLU, down projection and residual. No layer has a bias.

The non-linear client steps are plain float32 torch operations: they are
outside the masked-product path (the paper evaluates them locally on the
trusted side and does not specify kernels for them), and the same code
serves the secure forward and the plaintext float32 reference, so the two
differ only in how the four linear layers are evaluated.
"""
from __future__ import annotations

import math
from typing import Callable, Dict, List

import torch

from .secure_linear import SecureLinear

LINEARS = ("qkv", "o", "gate_up", "down")


def rms_norm(x: torch.Tensor, eps: float = 1e-5) -> torch.Tensor:
    return x * torch.rsqrt(x.pow(2).mean(dim=-1, keepdim=True) + eps)


def attention(qkv: torch.Tensor, cfg: dict) -> torch.Tensor:
    """Causal grouped-query attention on the fused q|k|v projection
    ((batch * seq) x (heads + 2 kv_heads) * head_dim), float32."""
    B, S = cfg["batch"], cfg["seq"]
    H, KV, D = cfg["heads"], cfg["kv_heads"], cfg["head_dim"]
    q = qkv[:, : H * D].reshape(B, S, H, D).transpose(1, 2).contiguous()
    k = qkv[:, H * D: (H + KV) * D].reshape(B, S, KV, D).transpose(1, 2)
    v = qkv[:, (H + KV) * D:].reshape(B, S, KV, D).transpose(1, 2)
    k = k.repeat_interleave(H // KV, dim=1).contiguous()
    v = v.repeat_interleave(H // KV, dim=1).contiguous()
    causal = torch.ones((S, S), dtype=torch.bool, device=qkv.device).triu_(1)
    out = torch.empty_like(q)
    for b in range(B):                       # one sequence at a time bounds the score memory
        s = torch.matmul(q[b], k[b].transpose(-1, -2).contiguous()) * (1.0 / math.sqrt(D))
        s.masked_fill_(causal, float("-inf"))
        out[b] = torch.matmul(torch.softmax(s, dim=-1), v[b])
    return out.transpose(1, 2).reshape(B * S, H * D).contiguous()


def block_forward(h: torch.Tensor, linear: Callable[[str, torch.Tensor], torch.Tensor], cfg: dict) -> torch.Tensor:
    """One decoder layer; ``linear(name, x)`` evaluates x W_name^T."""
    a = rms_norm(h).contiguous()
    h = h + linear("o", attention(linear("qkv", a), cfg))
    a = rms_norm(h).contiguous()
    gu = linear("gate_up", a)
    F = cfg["ffn"]
    act = (torch.nn.functional.silu(gu[:, :F]) * gu[:, F:]).contiguous()
    del gu
    return h + linear("down", act)


def plaintext_forward(x: torch.Tensor, weights: List[Dict[str, torch.Tensor]], cfg: dict) -> List[torch.Tensor]:
    """Float32 reference: hidden states after each layer."""
    outs, h = [], x
    for layer in weights:
        h = block_forward(h, lambda name, a, W=layer: torch.nn.functional.linear(a, W[name]), cfg)
        outs.append(h)
    return outs


class SecureDecoder:
    """The stack with every linear layer behind Pi_Sec-Linear. Layer l's
    linear i uses weight id 4 l + i; each forward uses fresh call ids."""

    def __init__(self, weights: List[Dict[str, torch.Tensor]], cfg: dict, params, seed: int):
        self.cfg = cfg
        self.layers = [{name: SecureLinear(layer[name], params, seed, weight_id=4 * li + i)
                        for i, name in enumerate(LINEARS)} for li, layer in enumerate(weights)]
        self.calls = 0

    def forward(self, x: torch.Tensor) -> List[torch.Tensor]:
        outs, h = [], x
        for layer in self.layers:
            def lin(name, a, L=layer):
                self.calls += 1
                return L[name](a, call_id=self.calls)
            h = block_forward(h, lin, self.cfg)
            outs.append(h)
        return outs


def error_metrics(got: torch.Tensor, ref: torch.Tensor) -> Dict[str, float]:
    """Relative l2 error and cosine similarity over the whole tensor (float64)."""
    g, r = got.double().flatten(), ref.double().flatten()
    rel = (g - r).norm() / r.norm()
    cos = torch.dot(g, r) / (g.norm() * r.norm())
    return {"rel_l2": float(rel), "cosine": float(cos)}
