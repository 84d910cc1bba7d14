"""Seeded synthetic inputs for the MOSAIC hot path.

This module is shared by the CPU oracle, the tests and the benchmark. It holds
only input generation (plaintext operands, activations, protocol parameter
sets); none of the method's arithmetic lives here.

Every generator uses ``numpy.random.default_rng(seed)`` and is deterministic.
Layouts follow the build convention: activations ``A`` are tokens x features
(M x K) and weights ``W`` are out-features x in-features (N x K), so the
plaintext product is ``A @ W.T`` (M x N). In the paper's notation
(Section 4, Y = W X with W m x n and X n x l) this is ``A = X^T``, ``W = W``,
M = l, K = n, N = m.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Tuple

import numpy as np


# ---------------------------------------------------------------------------
# protocol parameter sets (data only)
# ---------------------------------------------------------------------------
@dataclass(frozen=True)
class NoiseSpec:
    """Distribution of the full-rank LWE error terms E_w and E_x.

    kind: "dgauss" (discrete Gaussian of parameter sigma, support [-bound, bound])
          or "zero" (no error term).
    """
    kind: str = "dgauss"
    sigma: float = 0.5
    bound: int = 4


@dataclass(frozen=True)
class ProtocolParams:
    """Parameters of the nested LWE/LPN mask (Section 4.2 protocol box).

    ranks: (r_1, ..., r_d); depth d = len(ranks); r_1 > r_2 > ... > r_d.
    sparse_log2_inv_density: the LPN masks S_i, T_i have density 2^-k.
    lpn_weights: (t_2, ..., t_d), the fixed row Hamming weight of S_{i+1}
        and of each token's row of T_{i+1}; empty means the density rule.
    noise: the LWE error E_w / E_x.
    """
    ranks: Tuple[int, ...] = (128,)
    noise: NoiseSpec = field(default_factory=NoiseSpec)
    sparse_log2_inv_density: int = 6
    lpn_weights: Tuple[int, ...] = ()

    @property
    def depth(self) -> int:
        return len(self.ranks)


# Depth-1 (LWE only) with small noise, as in the deployed parameterisation.
PARAMS_D1_SMALL_R128 = ProtocolParams(ranks=(128,), noise=NoiseSpec("dgauss", 0.5, 4))
# Depth-2 (LWE + one LPN level), sparse masks at density 1/64 and no E.
PARAMS_D2_SPARSE = ProtocolParams(ranks=(128, 64), noise=NoiseSpec("zero", 0.0, 0))
# Depth-3 with sparse masks and small noise.
PARAMS_D3_SPARSE_SMALL = ProtocolParams(ranks=(192, 128, 64), noise=NoiseSpec("dgauss", 0.5, 4))
# The paper's LWE rank at lambda = 140 (r_1 = 1536, sigma = 0.5), depth 1.
PARAMS_PAPER_D1 = ProtocolParams(ranks=(1536,), noise=NoiseSpec("dgauss", 0.5, 4))
# Depth 2 with the paper's first two ranks (1536, 1024), sparse, no E.
PARAMS_PAPER_D2_SPARSE = ProtocolParams(ranks=(1536, 1024), noise=NoiseSpec("zero", 0.0, 0))
# Depth 3 with the paper's ranks (1536, 1024, 652) (Section 4.2 example
# parameterisation), sparse levels at density 1/64, no E.
PARAMS_PAPER_D3_SPARSE = ProtocolParams(ranks=(1536, 1024, 652), noise=NoiseSpec("zero", 0.0, 0))
# Example 4.1 in full: LWE r_1 = 1536 with sigma = 0.5, LPN-1 r_2 = 1024 and
# LPN-2 r_3 = 652, both with row Hamming weight t = 80.
PARAMS_PAPER_D3_T80 = ProtocolParams(ranks=(1536, 1024, 652), noise=NoiseSpec("dgauss", 0.5, 4),
                                     lpn_weights=(80, 80))
# Depth 2 with the paper's first two levels (r_2 = 1024, t_2 = 80) and sigma = 0.5.
PARAMS_PAPER_D2_T80 = ProtocolParams(ranks=(1536, 1024), noise=NoiseSpec("dgauss", 0.5, 4),
                                     lpn_weights=(80,))
# Decode workload rerun with the paper's small LWE error (sigma = 0.5) on
# top of the depth-2 sparse masks (density 2^-6).
PARAMS_DECODE_D2_NOISY = ProtocolParams(ranks=(1536, 1024), noise=NoiseSpec("dgauss", 0.5, 4))
# Small fixed-weight instance for parity at the single-matmul size.
PARAMS_D3_WEIGHT_SMALL = ProtocolParams(ranks=(192, 128, 64), noise=NoiseSpec("dgauss", 0.5, 4),
                                        lpn_weights=(12, 9))


# ---------------------------------------------------------------------------
# plaintext operands
# ---------------------------------------------------------------------------
def int8_operands(M: int, K: int, N: int, seed: int) -> Tuple[np.ndarray, np.ndarray]:
    """Uniform int8 plaintext in [-127, 127]: A (M x K) first, then W (N x K)."""
    rng = np.random.default_rng(seed)
    A = rng.integers(-127, 128, size=(M, K), dtype=np.int8)
    W = rng.integers(-127, 128, size=(N, K), dtype=np.int8)
    return A, W


def int8_matrix(rows: int, cols: int, seed: int) -> np.ndarray:
    rng = np.random.default_rng(seed)
    return rng.integers(-127, 128, size=(rows, cols), dtype=np.int8)


def outlier_activations(rows: int, n: int, seed: int, p_outlier: float = 1e-3,
                        scale: float = 50.0) -> np.ndarray:
    """fp32 activations: N(0, 1) entries, each independently an outlier with
    probability ``p_outlier``, outliers multiplied by ``scale``."""
    rng = np.random.default_rng(seed)
    x = rng.standard_normal((rows, n))
    mask = rng.random((rows, n)) < p_outlier
    x = np.where(mask, x * scale, x)
    return x.astype(np.float32)


# ---------------------------------------------------------------------------
# workload shapes
# ---------------------------------------------------------------------------
# Single masked matmul: A 64 x 512, W 512 x 512 (seed 0).
SMALL_CASE = dict(M=64, K=512, N=512, seed=0)
# Decode-shaped GEMMs at 8B-layer shapes (seed 1).
DECODE_M = (1, 8, 64)
DECODE_KN: List[Tuple[int, int]] = [(4096, 4096), (4096, 14336), (14336, 4096)]
DECODE_SEED = 1
# Prefill-shaped GEMMs at 70B-layer shapes (seed 2).
PREFILL_M = 2048
PREFILL_KN: List[Tuple[int, int]] = [(8192, 8192), (8192, 28672), (28672, 8192)]
PREFILL_SEED = 2
# Random-Hadamard rotation: 4096 x 8192 fp32, signs seed 3.
HADAMARD_SHAPE = (4096, 8192)
HADAMARD_SEED = 3

# Synthetic 70B-style decoder stack (end-to-end workload): hidden 8192,
# 64 query heads and 8 key/value heads of dimension 128, SwiGLU FFN 28672,
# 4 layers; weights N(0, 0.02^2); input hidden states N(0, 1) for batch 4 x
# sequence 1024 (seed 4).
DECODER = dict(hidden=8192, heads=64, kv_heads=8, head_dim=128, ffn=28672, layers=4, batch=4, seq=1024)
DECODER_SEED = 4
DECODER_WEIGHT_STD = 0.02
# linear layers of one block, in evaluation order; q|k|v and gate|up are
# single fused products (one masked activation per layer input)
DECODER_LINEARS = ("qkv", "o", "gate_up", "down")


def decoder_linear_shape(name: str, cfg: dict = DECODER) -> Tuple[int, int]:
    """(N, K) = (out features, in features) of one linear layer."""
    h, hd = cfg["hidden"], cfg["head_dim"]
    return {
        "qkv": ((cfg["heads"] + 2 * cfg["kv_heads"]) * hd, h),
        "o": (h, cfg["heads"] * hd),
        "gate_up": (2 * cfg["ffn"], h),
        "down": (h, cfg["ffn"]),
    }[name]


def decoder_weight(layer: int, name: str, device, cfg: dict = DECODER, seed: int = DECODER_SEED):
    """fp32 weight (N x K) ~ N(0, DECODER_WEIGHT_STD^2), from torch's
    generator on ``device`` seeded per (seed, layer, linear)."""
    import torch
    N, K = decoder_linear_shape(name, cfg)
    g = torch.Generator(device=device)
    g.manual_seed(seed * 1_000_003 + layer * 16 + DECODER_LINEARS.index(name))
    w = torch.randn((N, K), generator=g, device=device, dtype=torch.float32)
    return w.mul_(DECODER_WEIGHT_STD)


def decoder_input(device, cfg: dict = DECODER, seed: int = DECODER_SEED):
    """Input hidden states, (batch * seq) x hidden fp32 ~ N(0, 1)."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed * 1_000_003 + 999)
    return torch.randn((cfg["batch"] * cfg["seq"], cfg["hidden"]), generator=g, device=device,
                       dtype=torch.float32)


def int_codes(rows: int, cols: int, qmax: int, seed: int) -> np.ndarray:
    """Uniform integer codes in [-qmax, qmax] (int32)."""
    rng = np.random.default_rng(seed)
    return rng.integers(-qmax, qmax + 1, size=(rows, cols), dtype=np.int32)


# Ring products of the decoder stack at their own shapes (M = 4096 tokens):
# (K, N) of the fused QKV, the fused gate|up and the down projection (the
# output projection is the (8192, 8192) prefill shape).
DECODER_RING_KN: List[Tuple[int, int]] = [(8192, 10240), (8192, 57344), (28672, 8192)]
DECODER_RING_SEED = 5


# Secure mat-vec sweep (one token, square weights), seed 6.
MATVEC_N = (4096, 8192, 16384, 36864)
MATVEC_SEED = 6

# Client-overhead sweep (Section 7 outsourcing-efficiency figure, one token,
# mask initialisation batched over 512 invocations). The figure gives only
# each model's hidden size d; the matrix shapes are taken from the models'
# published configurations: the attention output projection (heads x head
# dimension -> d), the MLP up projection (d -> f) and the MLP down
# projection (f -> d), f the dense feed-forward width.
# (name, d, attention heads x head dimension, f)
OVERHEAD_MODELS = (
    ("LLaMA-3.2 1B", 2048, 2048, 8192),
    ("Gemma-2 27B", 4608, 4096, 36864),
    ("LLaMA-4 Maverick", 5120, 5120, 16384),
    ("Kimi-K2.5", 7168, 8192, 18432),
    ("DeepSeek-V3", 7168, 16384, 18432),
    ("LLaMA-3.1 70B", 8192, 8192, 28672),
    ("GPT-3 175B", 12288, 12288, 49152),
    ("LLaMA-3.1 405B", 16384, 16384, 53248),
)
OVERHEAD_BATCH = 512
OVERHEAD_SEED = 8


def int8_matrix_device(rows: int, cols: int, seed: int, device):
    """Uniform int8 in [-127, 127] drawn by torch's generator on ``device``
    (for matrices too large to draw on the host quickly)."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed)
    return torch.randint(-127, 128, (rows, cols), generator=g, device=device, dtype=torch.int8)
