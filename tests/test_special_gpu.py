"""IEEE special values through every kernel path (the output reading of the
paper's half-precision arithmetic: fp32 accumulation, one RNE rounding to
f16, overflow to +-inf, NaN propagating).

Planted on top of a seeded random case, against the oracle's binary64 sum:
* a NaN activation: its whole output row is NaN;
* a +inf activation: its row is +-inf where the weight is nonzero, NaN where
  it is zero, or NaN where +inf and -inf terms meet;
* a NaN scale and an infinite scale: the dequantized weights of that group
  become NaN / +-inf (NaN where q == z);
* one row of large activations against columns of all-positive and
  all-negative weights: outputs far beyond the f16 range, so +inf and -inf.
Which outputs are NaN, +inf, -inf or finite does not depend on the order of
the additions, so it is compared exactly; finite outputs to the usual bound."""
import numpy as np
import pytest

import oracle
import paper_2402_10076_amd as Q
from gpu_util import TOL, Packed, f16_values, from_dev_y, rand_case, say, to_dev_x

pytestmark = pytest.mark.gpu

F16_NAN, F16_INF, F16_NINF = 0x7E00, 0x7C00, 0xFC00
F16_OVERFLOW = 65520.0   # binary16 RNE: |v| >= 65520 rounds to infinity


def _case(M, K, N, seed):
    x, q, z, s = rand_case(seed, M, K, N)
    x[3, 5] = F16_NAN
    x[7, 100] = F16_INF
    s[2 % (K // 128), 10] = F16_NAN
    s[0, 20] = F16_INF
    # all-positive and all-negative weight columns, and a row of large activations
    q[:, 40], z[:, 40] = 15, 0
    q[:, 41], z[:, 41] = 0, 15
    s[:, 40:42] = np.float16(1.0).view(np.uint16)
    x[12, :] = np.float16(200.0).view(np.uint16)
    return x, q, z, s


def _classes(v):
    """0 finite, 1 NaN, 2 +inf, 3 -inf (a value at or beyond the f16 overflow
    bound counts as the infinity it rounds to)."""
    c = np.zeros(v.shape, np.int8)
    c[np.isnan(v)] = 1
    c[~np.isnan(v) & (v >= F16_OVERFLOW)] = 2
    c[~np.isnan(v) & (v <= -F16_OVERFLOW)] = 3
    return c


def _compare(y_bits, ref, what):
    y = f16_values(y_bits)
    cy, cr = _classes(y), _classes(ref)
    bad = np.argwhere(cy != cr)
    assert bad.size == 0, "%s: special-value class differs at %s (got %s, want %s)" % (
        what, bad[:5].tolist(), [y[tuple(i)] for i in bad[:5]], [ref[tuple(i)] for i in bad[:5]])
    fin = cr == 0
    err = np.max(np.abs(y[fin] - ref[fin])) / np.max(np.abs(ref[fin]))
    assert err <= TOL, "%s: finite outputs rel err %.3g" % (what, err)
    return int((cr == 1).sum()), int((cr >= 2).sum())


CFGS = [None, dict(variant=1, split_k=1, tile_n=1), dict(variant=1, split_k=4, tile_n=2),
        dict(variant=2, split_k=1, tile_m=16, tile_n=16), dict(variant=2, split_k=3, tile_m=32, tile_n=32),
        dict(variant=3, split_k=8, tile_m=16, tile_n=32), dict(variant=3, split_k=0, tile_m=128, tile_n=32),
        dict(variant=6, split_k=1, tile_m=32, tile_n=32), dict(variant=7, split_k=8, tile_m=64, tile_n=32)]


@pytest.mark.parametrize("cfg", CFGS, ids=lambda c: "auto" if c is None else "v%d_s%d_%dx%d" % (
    c["variant"], c["split_k"], c.get("tile_m", 0), c["tile_n"]))
@pytest.mark.parametrize("M", [16, 40])
def test_special_values(M, cfg):
    K, N = 512, 96
    x, q, z, s = _case(M, K, N, 61 + M)
    ref = oracle.gemm(x, q, z, s)
    p = Packed(q, z, s)
    say("special values M=%d cfg=%s" % (M, cfg))
    y = from_dev_y(p.gemm(to_dev_x(x), cfg=Q.make_config(**cfg) if cfg else None))
    nans, infs = _compare(y, ref, "M=%d cfg=%s" % (M, cfg))
    assert nans >= N + M - 1 and infs >= 2   # the planted row and column, the overflowing pair


@pytest.mark.parametrize("S", [1, 2, 4])
def test_special_values_sliced(S):
    """The sliced stream kernel (M <= 16) and its cross-workgroup finish."""
    M, K, N = 16, 512, 96
    x, q, z, s = _case(M, K, N, 71)
    ref = oracle.gemm(x, q, z, s)
    p = Packed(q, z, s)
    say("special values sliced S=%d" % S)
    y = from_dev_y(p.gemm(to_dev_x(x), cfg=Q.make_config(variant=5, split_k=S, tile_n=1)))
    _compare(y, ref, "sliced S=%d" % S)
