"""Seeded synthetic inputs for the W4A16 GEMM workloads.

This module only draws random numbers and describes shapes.  It contains no
dequantization, no packing and no GEMM arithmetic, so both the CPU oracle side
(tests) and the GPU side (binding, bench) can take their inputs from it
without sharing any of the method's code.

Every tensor is drawn from a numpy ``PCG64`` generator seeded with
``(config_id, shape_index, stream)`` so any single shape can be regenerated on
its own.  Distributions follow the workload definitions:

* x : fp16 = round-to-nearest-even of N(0, 1), shape [M][K]
      (Llama-2-13B set: floor(0.01*K) distinct input channels scaled by 20
      before rounding, to mimic activation outlier channels)
* q : uint4 uniform in 0..15, stored one value per uint8, shape [K][N]
* z : uint4 uniform in 0..15, shape [K/128][N]
* s : fp16 = RNE of U[0.002, 0.02], shape [K/128][N]

The shapes are the public decoder-linear dimensions of Llama-2-7B, -13B,
-70B and Mixtral-8x7B; no weights or datasets are used.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

GROUP = 128


@dataclass(frozen=True)
class Shape:
    name: str
    K: int
    N: int
    Ms: tuple


@dataclass(frozen=True)
class Config:
    cid: int
    name: str
    shapes: tuple
    outliers: bool = False
    desc: str = ""


C1 = Config(1, "toy-16x512x512", (Shape("toy", 512, 512, (16,)),),
            desc="single GEMM M=16 K=512 N=512")
C2 = Config(2, "llama2-7b", (
    Shape("qkv", 4096, 12288, (1, 4, 16, 64, 128, 256)),
    Shape("o_proj", 4096, 4096, (1, 4, 16, 64, 128, 256)),
    Shape("gate_up", 4096, 22016, (1, 4, 16, 64, 128, 256)),
    Shape("down", 11008, 4096, (1, 4, 16, 64, 128, 256)),
), desc="Llama-2-7B decoder linears")
C3 = Config(3, "llama2-13b", (
    Shape("qkv", 5120, 15360, (1, 16, 64, 256, 512)),
    Shape("o_proj", 5120, 5120, (1, 16, 64, 256, 512)),
    Shape("gate_up", 5120, 27648, (1, 16, 64, 256, 512)),
    Shape("down", 13824, 5120, (1, 16, 64, 256, 512)),
), outliers=True, desc="Llama-2-13B decoder linears, 1% outlier channels x20")
C4 = Config(4, "mixtral-8x7b-experts", (
    Shape("w1", 4096, 14336, ()),
    Shape("w3", 4096, 14336, ()),
    Shape("w2", 14336, 4096, ()),
), desc="Mixtral-8x7B expert FFN, 8 experts, top-2 of 512 tokens")
C5 = Config(5, "llama2-70b", (
    Shape("qkv", 8192, 10240, (1, 16, 128, 512, 1024)),
    Shape("o_proj", 8192, 8192, (1, 16, 128, 512, 1024)),
    Shape("gate_up", 8192, 57344, (1, 16, 128, 512, 1024)),
    Shape("down", 28672, 8192, (1, 16, 128, 512, 1024)),
), desc="Llama-2-70B decoder linears (single GPU, unsharded)")

CONFIGS = {1: C1, 2: C2, 3: C3, 4: C4, 5: C5}

MIXTRAL_EXPERTS = 8
MIXTRAL_TOKENS = 512
MIXTRAL_TOPK = 2

# stream ids inside one (config, shape) seed
_X, _W, _OUT = 0, 1, 2


def rng(cid: int, shape_index: int, stream: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64([cid, shape_index, stream]))


def f16_bits(a: np.ndarray) -> np.ndarray:
    """Round float values to binary16 (numpy's RNE cast) and return the bits."""
    return np.ascontiguousarray(np.asarray(a, np.float64).astype(np.float16)).view(np.uint16)


def draw_x(cid: int, shape_index: int, M: int, K: int, outliers: bool = False) -> np.ndarray:
    """Activations [M][K] as binary16 bits.  Rows are drawn in order, so a
    smaller M gives the leading rows of a larger one."""
    g = rng(cid, shape_index, _X)
    x = g.standard_normal((M, K))
    if outliers:
        go = rng(cid, shape_index, _OUT)
        ch = go.choice(K, size=K // 100, replace=False)
        x[:, ch] *= 20.0
    return f16_bits(x)


def draw_weights(cid: int, shape_index: int, K: int, N: int, group: int = GROUP):
    """(q [K][N] u8, z [K/g][N] u8, s [K/g][N] binary16 bits)."""
    g = rng(cid, shape_index, _W)
    q = g.integers(0, 16, size=(K, N), dtype=np.uint8)
    z = g.integers(0, 16, size=(K // group, N), dtype=np.uint8)
    s = f16_bits(g.uniform(0.002, 0.02, size=(K // group, N)))
    return q, z, s


def shape_inputs(cfg: Config, shape_index: int, M: int):
    sh = cfg.shapes[shape_index]
    x = draw_x(cfg.cid, shape_index, M, sh.K, cfg.outliers)
    q, z, s = draw_weights(cfg.cid, shape_index, sh.K, sh.N)
    return x, q, z, s


def mixtral_routing(seed: int = 4):
    """Top-2 uniform routing of 512 tokens over 8 experts.

    Returns a list of 8 int64 arrays: the token indices routed to each expert,
    in token order."""
    g = np.random.Generator(np.random.PCG64([seed, 99, 0]))
    picks = np.stack([g.choice(MIXTRAL_EXPERTS, size=MIXTRAL_TOPK, replace=False)
                      for _ in range(MIXTRAL_TOKENS)])
    return [np.nonzero((picks == e).any(axis=1))[0].astype(np.int64)
            for e in range(MIXTRAL_EXPERTS)]


def mixtral_tokens(seed: int = 4) -> np.ndarray:
    """Token activations [512][4096] binary16 bits."""
    g = np.random.Generator(np.random.PCG64([seed, 98, 0]))
    return f16_bits(g.standard_normal((MIXTRAL_TOKENS, 4096)))


def mixtral_expert_weights(expert: int, which: int):
    """which: 0 = w1, 1 = w3 (K=4096, N=14336), 2 = w2 (K=14336, N=4096)."""
    sh = C4.shapes[which]
    return draw_weights(4, 10 + 3 * expert + which, sh.K, sh.N)


def mixtral_w2_input(expert: int, M: int) -> np.ndarray:
    """Fresh fp16 N(0,1) input [M][14336] for an expert's w2 GEMM."""
    g = np.random.Generator(np.random.PCG64([4, 200 + expert, 0]))
    return f16_bits(g.standard_normal((M, 14336)))


def sample_columns(N: int, n_sample: int = 1024, seed: int = 0) -> np.ndarray:
    """Column sample for large shapes: the first and last n_sample/4 columns
    and n_sample/2 random ones in between (sorted, distinct); all columns when
    N <= n_sample."""
    if N <= n_sample:
        return np.arange(N, dtype=np.int64)
    e = n_sample // 4
    g = np.random.Generator(np.random.PCG64([seed, N, 7]))
    head = np.arange(e)
    tail = np.arange(N - e, N)
    mid = g.choice(np.arange(e, N - e), size=n_sample - 2 * e, replace=False)
    return np.unique(np.concatenate([head, tail, mid])).astype(np.int64)


def sample_rows(M: int, n_sample: int = 64, seed: int = 0) -> np.ndarray:
    """Row sample: all rows when M <= n_sample, else the first and last
    n_sample/4 rows and n_sample/2 random ones in between."""
    if M <= n_sample:
        return np.arange(M, dtype=np.int64)
    e = n_sample // 4
    g = np.random.Generator(np.random.PCG64([seed, M, 11]))
    mid = g.choice(np.arange(e, M - e), size=n_sample - 2 * e, replace=False)
    return np.unique(np.concatenate([np.arange(e), np.arange(M - e, M), mid])).astype(np.int64)


def alg_bytes(M: int, N: int, K: int, group: int = GROUP) -> int:
    """Bytes the method must move: packed int4 weights, fp16 scales, uint4
    zeros, fp16 activations in and fp16 outputs out."""
    return K * N // 2 + 2 * N * (K // group) + N * (K // group) // 2 + 2 * M * K + 2 * M * N


def flops(M: int, N: int, K: int) -> int:
    return 2 * M * N * K
