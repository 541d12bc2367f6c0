"""Helpers for the GPU tests: run the HIP path through the C ABI binding on
host-generated inputs and measure the error against the oracle."""
from __future__ import annotations

import sys

import numpy as np
import torch

import paper_2402_10076_amd as Q

TOL = 5e-3  # max|y - y_ref| / max|y_ref|, fp16 output, fp32 accumulation


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def to_dev_x(x_bits: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(x_bits).view(np.int16)).to("cuda").view(torch.float16)


def from_dev_y(y: torch.Tensor) -> np.ndarray:
    return y.cpu().view(torch.int16).numpy().view(np.uint16)


def f16_values(bits: np.ndarray) -> np.ndarray:
    return np.asarray(bits, np.uint16).view(np.float16).astype(np.float64)


class Packed:
    def __init__(self, q, z, s):
        self.K, self.N = q.shape
        pw, ps, pz = Q.pack_weights(q, z, s)
        self.dw, self.ds, self.dz = Q.to_device(pw, ps, pz)

    def gemm(self, x_dev, cfg=None, y=None, workspace=None, stream=None):
        return Q.w4a16_gemm(x_dev, self.dw, self.ds, self.dz, self.N, y=y, cfg=cfg,
                            workspace=workspace, stream=stream)


def run(x_bits, q, z, s, cfg=None) -> np.ndarray:
    """y bits (uint16 [M][N]) from the GPU."""
    p = Packed(q, z, s)
    y = p.gemm(to_dev_x(x_bits), cfg=cfg)
    torch.cuda.synchronize()
    return from_dev_y(y)


def rel_err(y_bits: np.ndarray, y_ref: np.ndarray) -> float:
    y = f16_values(y_bits)
    assert np.all(np.isfinite(y)), "non-finite output"
    den = np.max(np.abs(y_ref))
    num = np.max(np.abs(y - y_ref)) if y.size else 0.0
    if den == 0:
        return 0.0 if num == 0 else float("inf")
    return float(num / den)


def rand_case(seed, M, K, N, outliers=False):
    g = np.random.Generator(np.random.PCG64(seed))
    xv = g.standard_normal((M, K))
    if outliers:
        ch = g.choice(K, size=max(1, K // 100), replace=False)
        xv[:, ch] *= 20
    x = xv.astype(np.float16).view(np.uint16)
    q = g.integers(0, 16, (K, N), dtype=np.uint8)
    z = g.integers(0, 16, (K // 128, N), dtype=np.uint8)
    s = g.uniform(0.002, 0.02, (K // 128, N)).astype(np.float16).view(np.uint16)
    return x, q, z, s


def decode_qpk16_tile(pw_words: np.ndarray, pz_words: np.ndarray, ps_halves: np.ndarray, K: int):
    """(q [K][16], z [K/128][16], s bits [K/128][16]) of one n-tile from its
    QPK16 words: the tile's K/128 units of 64 lanes x 4 words (lane 16g + c,
    word j holds channels 32j + 8g + e of column c, element e in nibble slot
    e/2 + 4(e%2)), its 2 zero words per k-group (column c in nibble c%8 of
    word c/8) and its 16 scale halves per k-group.  Test infrastructure: the
    tests check it against the oracle's pack, which defines the layout."""
    KG = K // 128
    w = np.asarray(pw_words, np.uint32).reshape(KG, 4, 16, 4)          # kg, g, c, j
    q = np.empty((KG, 4, 4, 8, 16), np.uint8)                           # kg, j, g, e, c
    for slot in range(8):
        e = 2 * (slot % 4) + slot // 4
        q[:, :, :, e, :] = ((w >> np.uint32(4 * slot)) & np.uint32(15)).transpose(0, 3, 1, 2)
    zw = np.asarray(pz_words, np.uint32).reshape(KG, 2, 1)
    z = ((zw >> (4 * np.arange(8, dtype=np.uint32))) & np.uint32(15)).reshape(KG, 16).astype(np.uint8)
    return q.reshape(K, 16), z, np.asarray(ps_halves, np.uint16).reshape(KG, 16).copy()
