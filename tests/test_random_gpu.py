"""Seeded random shapes under random explicit configurations (plain, grouped
and fused-epilogue forms): every kernel,
tile, split and schedule the library accepts, on shapes with ragged M and
N tails, checked element by element against the oracle.  A configuration
the library rejects must be rejected with INVALID_ARG and is counted."""
import numpy as np
import pytest

import oracle
import paper_2402_10076_amd as Q
from gpu_util import TOL, Packed, from_dev_y, rand_case, rel_err, say, to_dev_x

pytestmark = pytest.mark.gpu

TILES = ((16, 16), (16, 32), (32, 16), (32, 32), (64, 16), (64, 32), (128, 16), (128, 32))
TILES32 = ((32, 32), (64, 32), (128, 32))


def _random_cfg(g, M, K):
    v = int(g.choice([0, 1, 2, 3, 5, 6, 7]))
    if v == 0:
        return None
    if v == 1:
        return dict(variant=1, split_k=int(g.choice([1, 2, 4, 8])), tile_n=int(g.choice([1, 2])))
    if v == 5:
        return dict(variant=5, split_k=int(g.integers(0, K // 128 + 1)), tile_n=int(g.choice([1, 2])))
    bm, wn = (TILES32 if v in (6, 7) else TILES)[int(g.integers(0, len(TILES32 if v in (6, 7) else TILES)))]
    if v in (3, 7):
        sk = int(g.choice([0, 8, 16, 24, 64, 256]))
    else:
        sk = int(g.integers(1, min(8, K // 128) + 1))
    return dict(variant=v, tile_m=bm, tile_n=wn, split_k=sk)


@pytest.mark.parametrize("seed", range(16))
def test_random_shapes_and_configs(seed):
    g = np.random.Generator(np.random.PCG64(9000 + seed))
    ran = rejected = 0
    for case in range(20):
        M = int(g.choice([1, 2, 3, 7, 16, 17, 33, 64, 65, 100, 128, 129]))
        K = 128 * int(g.integers(1, 17))
        N = 16 * int(g.integers(1, 65))
        x, q, z, s = rand_case(int(g.integers(1 << 30)), M, K, N)
        p = Packed(q, z, s)
        xd = to_dev_x(x)
        ref = oracle.gemm(x, q, z, s)
        for _ in range(3):
            cfg = _random_cfg(g, M, K)
            say("random seed=%d case=%d M=%d K=%d N=%d cfg=%s" % (seed, case, M, K, N, cfg))
            try:
                y = from_dev_y(p.gemm(xd, cfg=Q.make_config(**cfg) if cfg else None))
            except Q.QuickError as e:
                assert e.status == Q.QUICK_ERR_INVALID_ARG, (cfg, e)
                rejected += 1
                continue
            assert rel_err(y, ref) <= TOL, (M, K, N, cfg)
            ran += 1
    say("random seed=%d: %d runs, %d rejected configurations" % (seed, ran, rejected))
    assert ran >= 40


GROUPED_TILES = ((16, 16), (16, 32), (32, 16), (32, 32), (64, 32), (128, 32))


@pytest.mark.parametrize("seed", range(8))
def test_random_grouped(seed):
    """The grouped form on random expert counts (empty experts and one-row
    experts included), random token routing and random explicit
    configurations, against the oracle's grouped GEMM."""
    from test_grouped_gpu import Grouped, _experts, _routing
    g = np.random.Generator(np.random.PCG64(7000 + seed))
    ran = 0
    for case in range(6):
        E = int(g.integers(1, 9))
        K = 128 * int(g.integers(1, 9))
        N = 16 * int(g.integers(1, 33))
        T = int(g.integers(1, 200))
        counts = [int(c) for c in g.choice([0, 1, 2, 15, 16, 17, 63, 64, 65, 127, 128, 129, 150], size=E)]
        rows, offsets = _routing(int(g.integers(1 << 30)), T, E, counts=counts)
        experts = _experts(int(g.integers(1 << 30)), E, K, N)
        x = rand_case(int(g.integers(1 << 30)), T, K, 16)[0]
        ref = oracle.grouped_gemm(x, rows, offsets, experts)
        gp = Grouped(experts)
        xd = to_dev_x(x)
        for _ in range(3):
            v = int(g.choice([0, 2, 3]))
            if v == 0:
                cfg = None
            else:
                bm, wn = GROUPED_TILES[int(g.integers(0, len(GROUPED_TILES)))]
                sk = int(g.integers(1, min(4, K // 128) + 1)) if v == 2 else int(g.choice([0, 8, 64]))
                cfg = dict(variant=v, tile_m=bm, tile_n=wn, split_k=sk)
            say("random grouped seed=%d case=%d E=%d T=%d K=%d N=%d counts=%s cfg=%s" % (
                seed, case, E, T, K, N, counts, cfg))
            y = from_dev_y(gp.run(xd, rows, offsets, cfg=Q.make_config(**cfg) if cfg else None))
            if offsets[-1]:
                assert rel_err(y, ref) <= TOL, (E, counts, cfg)
            ran += 1
    assert ran == 18


@pytest.mark.parametrize("seed", range(6))
def test_random_fused_epilogues(seed):
    """Bias and the gated SiLU on random shapes and random explicit
    configurations, against the oracle's GEMM and binary64 epilogue; a
    configuration that cannot pair gate and up tiles in one wave is
    INVALID_ARG."""
    from test_fused_gpu import _bias, _dev_bias, _gate_up
    g = np.random.Generator(np.random.PCG64(5000 + seed))
    ran = 0
    for case in range(8):
        M = int(g.choice([1, 5, 16, 17, 64, 65, 130]))
        K = 128 * int(g.integers(1, 13))
        Nh = 16 * int(g.integers(1, 33))
        act = int(g.integers(0, 2))
        if act:
            q, z, s = _gate_up(int(g.integers(1 << 30)), K, Nh)
        else:
            _, q, z, s = rand_case(int(g.integers(1 << 30)), 1, K, Nh)
        N = q.shape[1]
        x = rand_case(int(g.integers(1 << 30)), M, K, 16)[0]
        b = _bias(int(g.integers(1 << 30)), N)
        dw, ds, dz = Q.to_device(*Q.pack_weights(q, z, s))
        ref = oracle.epilogue(oracle.gemm(x, q, z, s), b, act=act)
        xd = to_dev_x(x)
        for _ in range(3):
            cfg = _random_cfg(g, M, K)
            say("random fused seed=%d case=%d M=%d K=%d N=%d act=%d cfg=%s" % (seed, case, M, K, N, act, cfg))
            try:
                y = from_dev_y(Q.gemm_fused(xd, dw, ds, dz, N, bias=_dev_bias(b), activation=act,
                                            cfg=Q.make_config(**cfg) if cfg else None))
            except Q.QuickError as e:
                assert e.status == Q.QUICK_ERR_INVALID_ARG, (cfg, e)
                continue
            assert y.shape == (M, N // 2 if act else N)
            assert rel_err(y, ref) <= TOL, (M, K, N, act, cfg)
            ran += 1
    assert ran >= 10
