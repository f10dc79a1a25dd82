"""Seeded synthetic inputs shared by the tests, the smoke check and the benchmark.

This module holds no arithmetic of the method: it only draws normal random
tensors with fixed seeds, on the CPU with torch's own generator, so that the
GPU path and the CPU oracle receive the same bits.

Workloads stand in for the paper's BERT-base layers (Section 6.1: a
768 x 3072 x 4096 feed-forward GEMM, and batch 8 x sequence 512 inference);
no trained weights or datasets are used.  Weights are N(0, 0.02^2) (BERT's
initialiser scale), activations N(0, 1).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import torch

W_STD = 0.02
X_STD = 1.0


def seed_for(workload: int, layer: int, which: str) -> int:
    """Seed of tensor ``which`` ('W' or 'X') of ``layer`` in ``workload``."""
    return 1000 * workload + 10 * layer + {"W": 0, "X": 1}[which]


def normal(shape, seed: int, std: float = 1.0, dtype=torch.float32) -> torch.Tensor:
    """A CPU tensor of N(0, std^2) draws (binary32, then cast to ``dtype``)."""
    gen = torch.Generator(device="cpu").manual_seed(int(seed))
    t = torch.randn(tuple(shape), generator=gen, dtype=torch.float32)
    if std != 1.0:
        t = t * std
    return t.to(dtype).contiguous()


@dataclass(frozen=True)
class Linear:
    """One sparse linear layer Y = W_s X: W is M x K, X is K x N."""
    M: int
    K: int
    N: int
    n: int
    m: int
    g: int
    dtype: torch.dtype = torch.float32
    name: str = ""

    @property
    def nnz(self) -> int:
        C = -(-self.K // self.m)
        return self.M * C * self.n

    @property
    def useful_flop(self) -> int:
        return 2 * self.N * self.nnz


@dataclass(frozen=True)
class Workload:
    key: str
    description: str
    layers: tuple = field(default_factory=tuple)


# Single 768x768 layer at 2:4 with groups of 4 rows; 128 tokens.
SINGLE_768 = Workload("single-768x768-2:4:4", "one 768x768 fp32 layer, 2:4, g=4, 128 tokens",
                      (Linear(768, 768, 128, 2, 4, 4, name="single"),))
# BERT-base FFN up-projection, 75% sparse: W 3072x768, 1:4, g=8, 32x128 tokens.
FFN_UP = Workload("bert-ffn-up-3072x768-1:4:8", "BERT-base FFN up-projection, fp32, 1:4 (75%), g=8, "
                  "4096 tokens", (Linear(3072, 768, 4096, 1, 4, 8, name="ffn_up"),))
# BERT-base FFN down-projection, 90% sparse: W 768x3072, 1:10, g=16.
FFN_DOWN = Workload("bert-ffn-down-768x3072-1:10:16", "BERT-base FFN down-projection, fp32, 1:10 (90%), "
                    "g=16, 4096 tokens", (Linear(768, 3072, 4096, 1, 10, 16, name="ffn_down"),))

BERT_HIDDEN = 768
BERT_FFN = 3072
BERT_LAYERS = 12
BERT_TOKENS = 8 * 512


def bert_stack_layers(tokens: int = BERT_TOKENS, n: int = 2, m: int = 8, g: int = 8):
    """The four projections of one BERT-base encoder layer (fp16, 2:8:8)."""
    h, f = BERT_HIDDEN, BERT_FFN
    return (Linear(3 * h, h, tokens, n, m, g, torch.float16, "qkv"),
            Linear(h, h, tokens, n, m, g, torch.float16, "ao"),
            Linear(f, h, tokens, n, m, g, torch.float16, "up"),
            Linear(h, f, tokens, n, m, g, torch.float16, "down"))


BERT_STACK = Workload("bert-base-linear-stack-12x-2:8:8-fp16",
                      "12 BERT-base encoder layers of sparse linears (QKV, attention-out, FFN up, "
                      "FFN down), fp16, 2:8:8, 4096 tokens", bert_stack_layers())

SWEEP_NM = ((2, 4), (1, 4), (2, 8), (1, 10), (1, 20))
SWEEP_G = (1, 4, 8, 16, 32)


def sweep_layers(N: int = 4096):
    """The n:m x g sweep on the 3072x768 FFN shape, plus the dense control."""
    out = [Linear(3072, 768, N, n, m, g, name=f"{n}:{m}:{g}") for n, m in SWEEP_NM for g in SWEEP_G]
    out.append(Linear(3072, 768, N, 4, 4, 1, name="dense-4:4:1"))
    return tuple(out)


SWEEP = Workload("sweep-3072x768", "n:m in {2:4,1:4,2:8,1:10,1:20} x g in {1,4,8,16,32} + dense, "
                 "fp32, 4096 tokens", sweep_layers())

WORKLOADS = {1: SINGLE_768, 2: FFN_UP, 3: FFN_DOWN, 4: BERT_STACK, 5: SWEEP}


def layer_inputs(workload: int, layer: int, lin: Linear, device="cpu"):
    """W (M x K) and X (K x N) for one layer of a workload, seeded."""
    W = normal((lin.M, lin.K), seed_for(workload, layer, "W"), W_STD, lin.dtype)
    X = normal((lin.K, lin.N), seed_for(workload, layer, "X"), X_STD, lin.dtype)
    return W.to(device), X.to(device)
