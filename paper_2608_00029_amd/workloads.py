"""Seeded synthetic inputs for the attention, loss-head and memory-bound
operator workloads.

This module only draws random numbers; it holds none of the operators'
arithmetic, and both the HIP path's callers and the CPU reference's callers
take their inputs from here.

Attention recipe (identical for every caller): a CPU ``torch.Generator`` seeded with
``seed`` draws float32 ``randn`` tensors of shape [B, H, S, D] in the order
Q, K, V, dO; Q and K are then multiplied by ``qk_sigma``; for bf16 workloads
every tensor is rounded to bfloat16 (round-to-nearest-even, torch's ``.to``).
The values stand in for the attention activations of GPT-2 124M training
(12 heads of dimension 64 at a 1024-token context, the model of the paper's
Table 4, at the batch of 8 sequences its section 6.1 says it trains with);
the paper's training data is not used.  The loss-head and memory-bound
operator generators below state their own recipes.
"""

from __future__ import annotations

import math
from dataclasses import dataclass

import torch


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    H: int
    S: int
    D: int
    scale: float
    dtype: str          # "f32" or "bf16": storage dtype of Q, K, V, O, dO, dQ, dK, dV
    qk_sigma: float     # standard deviation of Q and K entries
    seed: int
    causal: bool = True

    @property
    def torch_dtype(self) -> torch.dtype:
        return torch.float32 if self.dtype == "f32" else torch.bfloat16

    @property
    def pairs(self) -> int:
        """Number of (query, key) pairs the mask keeps, summed over B*H."""
        per_head = self.S * (self.S + 1) // 2 if self.causal else self.S * self.S
        return self.B * self.H * per_head

    def counted_flops(self) -> tuple[float, float]:
        """Causal FLOP count used for throughput: fwd 2*B*H*S^2*D, bwd 5*B*H*S^2*D
        (half of the dense 4*B*H*S^2*D and 10*B*H*S^2*D); dense counts when not causal."""
        base = self.B * self.H * self.S * self.S * self.D
        f = 1.0 if self.causal else 2.0
        return 2.0 * base * f, 5.0 * base * f


SEED_BASE = 1234

WORKLOADS = [
    Workload("tiny_f32_B1_H2_S128_D64", 1, 2, 128, 64, 1.0 / 8.0, "f32", 1.0, SEED_BASE + 0),
    Workload("gpt2_small_B8_H12_S1024_D64", 8, 12, 1024, 64, 1.0 / 8.0, "bf16", 1.0, SEED_BASE + 1),
    Workload("gpt2_medium_B8_H16_S1024_D64", 8, 16, 1024, 64, 1.0 / 8.0, "bf16", 1.0, SEED_BASE + 2),
    Workload("gpt2_xl_width_B4_H25_S1024_D64", 4, 25, 1024, 64, 1.0 / 8.0, "bf16", 1.0, SEED_BASE + 3),
    Workload("long_ctx_B2_H16_S4096_D128", 2, 16, 4096, 128, 1.0 / math.sqrt(128.0), "bf16", 3.0,
             SEED_BASE + 4),
]

# Shapes of the kind the paper's attention sweep covers (sequence lengths 512,
# 1024 and 2048, 12 to 32 heads, head dimension 64 or 128; section 6, attention
# benchmark), at the batch of 16 its attention microbenchmark uses.  The paper
# prints its per-shape results only as figures, so these are representative
# points of that range, not its exact list; B16 H12 S1024 D64 is the shape of
# its fused-attention latency figure.  Timed by the benchmark after its timed
# region and parity-checked on sampled heads, like the workloads above.
SWEEP = [
    Workload("sweep_B16_H12_S512_D64", 16, 12, 512, 64, 1.0 / 8.0, "bf16", 1.0, SEED_BASE + 10),
    Workload("sweep_B16_H12_S1024_D64", 16, 12, 1024, 64, 1.0 / 8.0, "bf16", 1.0, SEED_BASE + 11),
    Workload("sweep_B16_H12_S2048_D64", 16, 12, 2048, 64, 1.0 / 8.0, "bf16", 1.0, SEED_BASE + 12),
    Workload("sweep_B16_H32_S1024_D64", 16, 32, 1024, 64, 1.0 / 8.0, "bf16", 1.0, SEED_BASE + 13),
    Workload("sweep_B16_H16_S512_D128", 16, 16, 512, 128, 1.0 / math.sqrt(128.0), "bf16", 1.0, SEED_BASE + 14),
    Workload("sweep_B16_H16_S1024_D128", 16, 16, 1024, 128, 1.0 / math.sqrt(128.0), "bf16", 1.0, SEED_BASE + 15),
]

BY_NAME = {w.name: w for w in WORKLOADS + SWEEP}


def make_inputs(B: int, H: int, S: int, D: int, dtype: str = "bf16", seed: int = SEED_BASE,
                qk_sigma: float = 1.0):
    """Return (q, k, v, do) CPU tensors, contiguous [B, H, S, D], in the storage dtype."""
    g = torch.Generator(device="cpu").manual_seed(seed)
    shape = (B, H, S, D)
    q = torch.randn(shape, generator=g, dtype=torch.float32)
    k = torch.randn(shape, generator=g, dtype=torch.float32)
    v = torch.randn(shape, generator=g, dtype=torch.float32)
    do = torch.randn(shape, generator=g, dtype=torch.float32)
    if qk_sigma != 1.0:
        q = q * qk_sigma
        k = k * qk_sigma
    td = torch.float32 if dtype == "f32" else torch.bfloat16
    return tuple(t.to(td).contiguous() for t in (q, k, v, do))


def workload_inputs(w: Workload):
    return make_inputs(w.B, w.H, w.S, w.D, w.dtype, w.seed, w.qk_sigma)


@dataclass(frozen=True)
class LmheadWorkload:
    """Fused loss-head shape: M tokens of hidden size K against an N-entry vocabulary."""
    name: str
    M: int
    N: int
    K: int
    w_sigma: float
    seed: int


# GPT-2 124M's head as the paper trains and measures it: 8 sequences of 1024
# tokens (M = 8192), hidden size 768, vocabulary 50257 padded to 50304.
LMHEAD_WORKLOADS = [
    LmheadWorkload("gpt2_lmhead_M8192_N50304_K768", 8192, 50304, 768, 0.02, SEED_BASE + 20),
]


def make_lmhead_inputs(M: int, N: int, K: int, w_sigma: float = 0.02, seed: int = SEED_BASE):
    """(x [M, K] bf16, w [N, K] bf16, targets [M] int32) CPU tensors: x ~ N(0, 1) (hidden states
    after the final normalisation), w ~ N(0, w_sigma^2) (GPT-2's embedding initialisation), targets
    uniform over the vocabulary.  Drawn in that order from one seeded CPU generator."""
    g = torch.Generator(device="cpu").manual_seed(seed)
    x = torch.randn((M, K), generator=g, dtype=torch.float32).to(torch.bfloat16)
    w = (torch.randn((N, K), generator=g, dtype=torch.float32) * w_sigma).to(torch.bfloat16)
    y = torch.randint(0, N, (M,), generator=g, dtype=torch.int64).to(torch.int32)
    return x.contiguous(), w.contiguous(), y.contiguous()


@dataclass(frozen=True)
class MemopsWorkload:
    """A memory-bound operator at the shape the paper measures it: LayerNorm over
    [rows, C], GELU over rows * C elements, softmax cross entropy over [rows, C]
    logits (C = vocabulary).  float32 tensors."""
    name: str
    op: str        # "layernorm", "gelu" or "sce"
    rows: int
    C: int
    seed: int


# The paper's memory-bound operator shapes (section 6, "Memory-Bound
# Operators"): 16 sequences of 1024 tokens with GPT-2's width 768 (LayerNorm),
# its MLP width 3072 (GELU) and its padded vocabulary 50304 (cross entropy).
MEMOPS_WORKLOADS = [
    MemopsWorkload("layernorm_16x1024x768", "layernorm", 16 * 1024, 768, SEED_BASE + 30),
    MemopsWorkload("gelu_16x1024x3072", "gelu", 16 * 1024, 3072, SEED_BASE + 31),
    MemopsWorkload("sce_16x1024x50304", "sce", 16 * 1024, 50304, SEED_BASE + 32),
]

GPT2_VOCAB = 50257  # real entries of the padded 50304-wide vocabulary


def make_layernorm_inputs(rows: int, C: int, seed: int = SEED_BASE):
    """(x [rows, C], gamma [C], beta [C], dy [rows, C]) float32 CPU tensors, drawn in that order:
    x ~ N(0, 1) + 0.5 (residual-stream activations with a row offset the mean removes),
    gamma ~ 1 + 0.1 N(0, 1), beta ~ 0.1 N(0, 1), dy ~ N(0, 1)."""
    g = torch.Generator(device="cpu").manual_seed(seed)
    x = torch.randn((rows, C), generator=g, dtype=torch.float32) + 0.5
    gamma = 1.0 + 0.1 * torch.randn((C,), generator=g, dtype=torch.float32)
    beta = 0.1 * torch.randn((C,), generator=g, dtype=torch.float32)
    dy = torch.randn((rows, C), generator=g, dtype=torch.float32)
    return x.contiguous(), gamma.contiguous(), beta.contiguous(), dy.contiguous()


def make_gelu_inputs(n: int, seed: int = SEED_BASE, sigma: float = 2.0):
    """(x [n], dy [n]) float32 CPU tensors: x ~ N(0, sigma^2) (MLP pre-activations; sigma 2 reaches
    both saturated tails of the tanh), dy ~ N(0, 1)."""
    g = torch.Generator(device="cpu").manual_seed(seed)
    x = torch.randn((n,), generator=g, dtype=torch.float32) * sigma
    dy = torch.randn((n,), generator=g, dtype=torch.float32)
    return x.contiguous(), dy.contiguous()


def make_sce_inputs(rows: int, V: int, seed: int = SEED_BASE, sigma: float = 2.0, n_real: int = 0):
    """(logits [rows, V] float32, targets [rows] int32) CPU tensors: logits ~ N(0, sigma^2), targets
    uniform over the first n_real entries (the real vocabulary; all V when n_real is 0)."""
    g = torch.Generator(device="cpu").manual_seed(seed)
    z = torch.randn((rows, V), generator=g, dtype=torch.float32) * sigma
    t = torch.randint(0, n_real or V, (rows,), generator=g, dtype=torch.int64).to(torch.int32)
    return z.contiguous(), t.contiguous()
