"""Seeded synthetic inputs and workload shapes for the DP-masked linear layer.

This module holds no arithmetic of the method: it only draws inputs (activations
X, weights W) with fixed seeds and names the projection shapes of the two model
families the paper evaluates (Sec. "Inference Models").  Both the oracle-side
tests and the GPU path take their inputs from here.

Recipe (the paper's Dolly prompts, real activations and trained weights are not
available; these stand in for them):
  X ~ N(0, 1) float32, rows = tokens;       numpy PCG64, seed ``x_seed``
  W ~ N(0, 0.02^2) drawn in float32, then rounded to bfloat16 by torch
    (float32 kept for the small float32 case); numpy PCG64, seed 2 + layer
  noise stream: seed 0, stream_id = (layer << 8) | group, row0 = 0 for prefill.
  normalisation scale alpha ~ N(1, 0.1^2), shift beta ~ N(0, 0.02^2), float32, d wide
    (stand-ins for trained values; alpha = 1, beta = 0 is the untrained layer)
"""
from dataclasses import dataclass, field
from typing import List

import numpy as np


@dataclass(frozen=True)
class Projection:
    """One masked GEMM group: inputs K wide, outputs N wide (fused where the
    paper shares one mask, Sec. "Precomputing the Mask and Noise Correction")."""
    name: str
    K: int
    N: int
    group: int  # stream-id group index


@dataclass(frozen=True)
class ModelShape:
    name: str
    layers: int
    hidden: int
    q_dim: int
    kv_dim: int
    ff: int
    vocab: int

    def lm_head(self) -> Projection:
        """The vocabulary projection after the final normalisation (offloaded too,
        Sec. "Inference Models"); its own noise group."""
        return Projection("lm_head", self.hidden, self.vocab, 4)

    def projections(self) -> List[Projection]:
        return [
            Projection("qkv", self.hidden, self.q_dim + 2 * self.kv_dim, 0),
            Projection("o", self.q_dim, self.hidden, 1),
            Projection("gate_up", self.hidden, 2 * self.ff, 2),
            Projection("down", self.ff, self.hidden, 3),
        ]


# Sec. "Inference Models": Llama-3.2-3B (28 layers, d 3072, d_ff 8192, 24 q / 8 kv
# heads of 128, vocabulary 128256) and Qwen3-4B (36 layers, d 2560, q 4096, k/v 1024,
# d_ff 9728, vocabulary 151936).
LLAMA_3B = ModelShape("llama-3.2-3b", 28, 3072, 3072, 1024, 8192, 128256)
QWEN3_4B = ModelShape("qwen3-4b", 36, 2560, 4096, 1024, 9728, 151936)


def stream_id(layer: int, group: int) -> int:
    return (layer << 8) | group


@dataclass(frozen=True)
class Workload:
    name: str
    model: ModelShape
    tokens: List[int]
    layers: int
    eps: List[float]
    mechs: List[str]
    w_dtype: str = "bf16"
    extra: dict = field(default_factory=dict)


# The five workloads: a single small float32 projection; one Llama layer at a
# 128-token prefill; the 28-layer Llama stack at 512 tokens; the 36-layer Qwen
# stack at 1024 tokens; Qwen decode steps against a 2048-position correction bank.
SINGLE_FP32 = dict(M=32, K=512, N=512, mech="laplace", delta=1.0, eps=1.0, seed=0)
LLAMA_LAYER_M128 = Workload("llama3b-layer-m128", LLAMA_3B, [128], 1, [1.0, 4.0, 16.0],
                            ["laplace", "gaussian"])
LLAMA_STACK_M512 = Workload("llama3b-28l-m512", LLAMA_3B, [512], 28, [0.5, 2.0, 8.0],
                            ["laplace", "gaussian"])
QWEN_STACK_M1024 = Workload("qwen3-4b-36l-m1024", QWEN3_4B, [1024], 36, [0.5, 2.0, 8.0],
                            ["laplace", "gaussian"])
QWEN_DECODE = Workload("qwen3-4b-decode", QWEN3_4B, [1, 4, 16, 64], 36, [0.5, 2.0, 8.0],
                       ["laplace", "gaussian"], extra=dict(bank_rows=2048))


def gen_x(M: int, K: int, seed: int = 1) -> np.ndarray:
    """Activations X ~ N(0, 1), float32, M x K."""
    return np.random.Generator(np.random.PCG64(seed)).standard_normal((M, K), dtype=np.float32)


def gen_w(N: int, K: int, seed: int = 2, std: float = 0.02, dtype: str = "bf16") -> np.ndarray:
    """Weights W ~ N(0, std^2), N x K (out x in).

    ``dtype='bf16'`` returns float32 values that are exactly bfloat16 (rounded by
    torch's float32 -> bfloat16 conversion); ``'f32'`` returns plain float32.
    """
    w = np.random.Generator(np.random.PCG64(seed)).standard_normal((N, K), dtype=np.float32)
    w = (w * np.float32(std)).astype(np.float32)
    if dtype == "f32":
        return w
    import torch
    return torch.from_numpy(w).to(torch.bfloat16).to(torch.float32).numpy()


def gen_norm(d: int, seed: int = 3, scale_std: float = 0.1, shift_std: float = 0.02):
    """Normalisation parameters (alpha, beta), float32, d wide."""
    g = np.random.Generator(np.random.PCG64(seed))
    alpha = (1.0 + scale_std * g.standard_normal(d)).astype(np.float32)
    beta = (shift_std * g.standard_normal(d)).astype(np.float32)
    return alpha, beta


def gen_int(shape, lo: int, hi: int, seed: int) -> np.ndarray:
    """Integer-valued float32 array, uniform on [lo, hi]."""
    g = np.random.Generator(np.random.PCG64(seed))
    return g.integers(lo, hi + 1, size=shape).astype(np.float32)


def bf16_upper_bits(w_bf16_valued: np.ndarray) -> np.ndarray:
    """The uint16 storage of float32 arrays whose values are exactly bfloat16."""
    b = np.ascontiguousarray(w_bf16_valued, dtype=np.float32).view(np.uint32)
    return (b >> np.uint32(16)).astype(np.uint16)
