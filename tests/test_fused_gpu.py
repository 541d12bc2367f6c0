"""Fused output epilogues (include/quick_fused.h) on the GPU through the C
ABI: bias and the gated SiLU of interleaved gate/up tiles, against the
oracle's GEMM followed by its binary64 epilogue, on every kernel path
(stream kernel, tiled data-parallel, split-K reduction, stream-K fix-up,
grouped)."""
import numpy as np
import pytest
import torch

import oracle
import paper_2402_10076_amd as Q
from gpu_util import TOL, from_dev_y, rand_case, rel_err, say, to_dev_x

pytestmark = pytest.mark.gpu


def _gate_up(seed, K, Nh):
    """Interleaved fused gate/up weights (q, z, s) of two random matrices."""
    g = np.random.Generator(np.random.PCG64(seed))

    def mat():
        return (g.integers(0, 16, (K, Nh), dtype=np.uint8), g.integers(0, 16, (K // 128, Nh), dtype=np.uint8),
                g.uniform(0.002, 0.02, (K // 128, Nh)).astype(np.float16).view(np.uint16))
    return Q.interleave_gate_up(mat(), mat())


def _bias(seed, n):
    g = np.random.Generator(np.random.PCG64(seed))
    return g.uniform(-2, 2, n).astype(np.float16).view(np.uint16)


def _dev_bias(b):
    return torch.from_numpy(b.view(np.int16)).cuda().view(torch.float16)


CFGS = [None,
        dict(variant=1, split_k=1, tile_n=2), dict(variant=1, split_k=4, tile_n=2),
        dict(variant=2, split_k=1, tile_m=16, tile_n=32), dict(variant=2, split_k=1, tile_m=64, tile_n=32),
        dict(variant=2, split_k=3, tile_m=32, tile_n=16), dict(variant=2, split_k=2, tile_m=128, tile_n=32),
        dict(variant=3, split_k=24, tile_m=32, tile_n=32), dict(variant=3, split_k=16, tile_m=128, tile_n=32),
        dict(variant=6, split_k=1, tile_m=64, tile_n=32), dict(variant=6, split_k=3, tile_m=32, tile_n=32),
        dict(variant=7, split_k=16, tile_m=128, tile_n=32)]


def _cid(c):
    return "auto" if c is None else "v%d_s%d_%dx%d" % (c["variant"], c["split_k"], c.get("tile_m", 0), c["tile_n"])


@pytest.mark.parametrize("cfg", CFGS, ids=_cid)
@pytest.mark.parametrize("M", [3, 70])
def test_gated_silu_with_bias(M, cfg):
    K, Nh = 1152, 144
    q, z, s = _gate_up(100 + M, K, Nh)
    N = 2 * Nh
    x = rand_case(200 + M, M, K, 16)[0]
    b = _bias(300 + M, N)
    dw, ds, dz = Q.to_device(*Q.pack_weights(q, z, s))
    say("gated M=%d cfg=%s" % (M, cfg))
    if cfg and cfg["variant"] == 1 and M > 64:
        # the stream kernel takes at most 64 rows: rejected before any launch
        with pytest.raises(Q.QuickError) as e:
            Q.gemm_fused(to_dev_x(x), dw, ds, dz, N, bias=_dev_bias(b), activation=Q.ACT_SILU_GATE,
                         cfg=Q.make_config(**cfg))
        assert e.value.status == Q.QUICK_ERR_INVALID_ARG
        return
    y = from_dev_y(Q.gemm_fused(to_dev_x(x), dw, ds, dz, N, bias=_dev_bias(b), activation=Q.ACT_SILU_GATE,
                                cfg=Q.make_config(**cfg) if cfg else None))
    assert y.shape == (M, Nh)
    ref = oracle.epilogue(oracle.gemm(x, q, z, s), b, act=1)
    err = rel_err(y, ref)
    say("  rel_err=%.3g" % err)
    assert err <= TOL


@pytest.mark.parametrize("cfg", [None, dict(variant=1, split_k=2, tile_n=1), dict(variant=2, split_k=2, tile_m=32,
                                 tile_n=16), dict(variant=3, split_k=8, tile_m=64, tile_n=32)], ids=_cid)
def test_bias_only(cfg):
    M, K, N = 33, 640, 80
    x, q, z, s = rand_case(41, M, K, N)
    b = _bias(42, N)
    dw, ds, dz = Q.to_device(*Q.pack_weights(q, z, s))
    say("bias cfg=%s" % cfg)
    c = Q.make_config(**cfg) if cfg else None
    y = from_dev_y(Q.gemm_fused(to_dev_x(x), dw, ds, dz, N, bias=_dev_bias(b), cfg=c))
    assert rel_err(y, oracle.epilogue(oracle.gemm(x, q, z, s), b)) <= TOL


def test_no_epilogue_is_the_plain_gemm_bitwise():
    """An empty epilogue leaves the GEMM's bits unchanged on the same plan."""
    M, K, N = 45, 1024, 208
    x, q, z, s = rand_case(51, M, K, N)
    dw, ds, dz = Q.to_device(*Q.pack_weights(q, z, s))
    xd = to_dev_x(x)
    for cfg in (None, Q.make_config(variant=2, split_k=3, tile_m=32, tile_n=16),
                Q.make_config(variant=3, split_k=8, tile_m=64, tile_n=32)):
        y0 = from_dev_y(Q.w4a16_gemm(xd, dw, ds, dz, N, cfg=cfg))
        y1 = from_dev_y(Q.gemm_fused(xd, dw, ds, dz, N, cfg=cfg))
        assert np.array_equal(y0, y1)


def test_grouped_gated_with_expert_bias():
    """Grouped GEMM over 4 experts of fused gate/up weights with a per-expert
    bias and the gated SiLU, gathered tokens; each expert's block against the
    oracle; data-parallel, stream-K and (activation only) split-K."""
    T, K, Nh, E = 40, 640, 112, 4
    experts = [_gate_up(60 + e, K, Nh) for e in range(E)]
    N = 2 * Nh
    x = rand_case(61, T, K, 16)[0]
    g = np.random.Generator(np.random.PCG64(62))
    counts = [23, 0, 57, 9]
    rows = np.concatenate([np.sort(g.integers(0, T, c)) for c in counts]).astype(np.int32)
    offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    bias = np.stack([_bias(70 + e, N) for e in range(E)])
    dw, ds, dz = Q.to_device(*Q.pack_experts(experts))
    od, rd = torch.from_numpy(offsets).cuda(), torch.from_numpy(rows).cuda()
    xd = to_dev_x(x)
    for cfg, with_bias in ((None, True), (Q.make_config(variant=2, split_k=1, tile_m=32, tile_n=32), True),
                           (Q.make_config(variant=3, split_k=16, tile_m=64, tile_n=32), True),
                           (Q.make_config(variant=2, split_k=3, tile_m=16, tile_n=16), False)):
        say("grouped gated cfg=%s bias=%s" % (cfg and cfg.as_dict(), with_bias))
        y = from_dev_y(Q.grouped_gemm_fused(xd, od, dw, ds, dz, N, rows=rd,
                                            bias=_dev_bias(bias.reshape(-1)) if with_bias else None,
                                            activation=Q.ACT_SILU_GATE, cfg=cfg))
        assert y.shape == (int(offsets[-1]), Nh)
        for e in range(E):
            lo, hi = offsets[e], offsets[e + 1]
            if hi == lo:
                continue
            ref = oracle.epilogue(oracle.gemm(x[rows[lo:hi]], *experts[e]), bias[e] if with_bias else None, act=1)
            assert rel_err(y[lo:hi], ref) <= TOL, "expert %d" % e


def test_grouped_gated_auto_two_parts():
    """Per-expert bias and the gated SiLU through the automatic two-launch
    plan (about 128 rows per expert: 128-row tiles, then 32-row tiles over
    the short remainders)."""
    T, K, Nh = 300, 512, 128
    counts = [131, 0, 127, 150, 100]
    E = len(counts)
    experts = [_gate_up(90 + e, K, Nh) for e in range(E)]
    N = 2 * Nh
    x = rand_case(91, T, K, 16)[0]
    g = np.random.Generator(np.random.PCG64(92))
    rows = np.concatenate([np.sort(g.integers(0, T, c)) for c in counts]).astype(np.int32)
    offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    bias = np.stack([_bias(93 + e, N) for e in range(E)])
    assert Q.grouped_select_config(int(offsets[-1]), E, N, K)["tile_m"] == 128
    dw, ds, dz = Q.to_device(*Q.pack_experts(experts))
    say("grouped gated two parts")
    y = from_dev_y(Q.grouped_gemm_fused(to_dev_x(x), torch.from_numpy(offsets).cuda(), dw, ds, dz, N,
                                        rows=torch.from_numpy(rows).cuda(), bias=_dev_bias(bias.reshape(-1)),
                                        activation=Q.ACT_SILU_GATE))
    for e in range(E):
        lo, hi = offsets[e], offsets[e + 1]
        if hi == lo:
            continue
        ref = oracle.epilogue(oracle.gemm(x[rows[lo:hi]], *experts[e]), bias[e], act=1)
        assert rel_err(y[lo:hi], ref) <= TOL, "expert %d" % e
