"""The sliced stream kernel (variant 5: the 8 waves of a workgroup split the
columns, workgroups split K into slices staged in LDS, last-arriver sum of
the slices) on the GPU through the C ABI, against the CPU oracle: ragged
column groups, uneven and single-k-group slices, slice counts raised to the
minimum, run-to-run determinism with the internal and a caller workspace,
the fused epilogues, and rejected configurations."""
import numpy as np
import pytest
import torch

import oracle
import paper_2402_10076_amd as Q
from gpu_util import TOL, Packed, from_dev_y, rand_case, rel_err, say, to_dev_x

pytestmark = pytest.mark.gpu

# (K, N): 17 n-tiles (a partial column group for 1 and 2 n-tiles per wave);
# 18 k-groups (two slices of 9, or 6 of 3 with split_k 7); 48 k-groups over
# 528 columns; one k-group; 224 k-groups (14 slices of 16)
SHAPES = ((4096, 272), (2304, 80), (6144, 528), (128, 16), (28672, 48))
KS_CFGS = [dict(variant=5, split_k=s, tile_n=p) for p in (1, 2) for s in (0, 1, 3, 7)]


def _check(M, K, N, cfg, seed):
    say("case M=%d K=%d N=%d cfg=%s" % (M, K, N, cfg))
    x, q, z, s = rand_case(seed, M, K, N)
    p = Packed(q, z, s)
    y = from_dev_y(p.gemm(to_dev_x(x), cfg=Q.make_config(**cfg)))
    err = rel_err(y, oracle.gemm(x, q, z, s))
    assert err <= TOL, "rel err %.3g for M=%d K=%d N=%d cfg=%s" % (err, M, K, N, cfg)


@pytest.mark.parametrize("cfg", KS_CFGS, ids=lambda c: "s%d_p%d" % (c["split_k"], c["tile_n"]))
@pytest.mark.parametrize("M", [1, 3, 9, 16])
def test_kstream_variants(M, cfg):
    for i, (K, N) in enumerate(SHAPES):
        if cfg["split_k"] <= K // 128:
            _check(M, K, N, cfg, seed=M * 100 + i + 7 * cfg["split_k"] + cfg["tile_n"])


def test_kstream_outlier_channels():
    """Activations with 1% of the channels scaled x20 (the 13B-shaped inputs)."""
    M, K, N = 16, 5120, 160
    x, q, z, s = rand_case(31, M, K, N, outliers=True)
    p = Packed(q, z, s)
    for cfg in (dict(variant=5, split_k=0, tile_n=2), dict(variant=5, split_k=10, tile_n=1)):
        say("outliers cfg=%s" % cfg)
        y = from_dev_y(p.gemm(to_dev_x(x), cfg=Q.make_config(**cfg)))
        assert rel_err(y, oracle.gemm(x, q, z, s)) <= TOL


def test_kstream_deterministic_and_caller_workspace():
    """Slices summed in slice order: repeated calls give identical bits with
    the internal or a caller workspace, whose counters are left zero."""
    M, K, N = 16, 8192, 528
    x, q, z, s = rand_case(78, M, K, N)
    p = Packed(q, z, s)
    xd = to_dev_x(x)
    cfg = Q.make_config(variant=5, split_k=8, tile_n=1)
    nb = Q.workspace_bytes(M, N, K, cfg)
    assert nb > Q.WS_COUNTER_BYTES
    ws = torch.zeros(nb // 4 + 1, dtype=torch.int32, device="cuda")
    say("kstream determinism ws=%d" % nb)
    y0 = from_dev_y(p.gemm(xd, cfg=cfg))
    y1 = from_dev_y(p.gemm(xd, cfg=cfg, workspace=ws))
    y2 = from_dev_y(p.gemm(xd, cfg=cfg, workspace=ws))
    assert np.array_equal(y0, y1) and np.array_equal(y1, y2)
    assert int(ws[:Q.WS_COUNTER_BYTES // 4].abs().sum().item()) == 0
    assert rel_err(y0, oracle.gemm(x, q, z, s)) <= TOL
    # one slice needs no workspace
    assert Q.workspace_bytes(M, N, 2048, Q.make_config(variant=5, split_k=1, tile_n=2)) == 0


@pytest.mark.parametrize("split", [1, 4])
def test_kstream_fused_epilogues(split):
    """Bias and the gated SiLU of interleaved gate/up tiles, applied by the
    workgroup that stores y (the only one, or the last slice to arrive)."""
    M, K, Nh = 9, 1152, 144
    g = np.random.Generator(np.random.PCG64(500 + split))

    def mat():
        return (g.integers(0, 16, (K, Nh), dtype=np.uint8), g.integers(0, 16, (K // 128, Nh), dtype=np.uint8),
                g.uniform(0.002, 0.02, (K // 128, Nh)).astype(np.float16).view(np.uint16))
    q, z, s = Q.interleave_gate_up(mat(), mat())
    N = 2 * Nh
    x = rand_case(600 + split, M, K, 16)[0]
    b = g.uniform(-2, 2, N).astype(np.float16).view(np.uint16)
    bd = torch.from_numpy(b.view(np.int16)).cuda().view(torch.float16)
    dw, ds, dz = Q.to_device(*Q.pack_weights(q, z, s))
    xd = to_dev_x(x)
    say("kstream gated split=%d" % split)
    y = from_dev_y(Q.gemm_fused(xd, dw, ds, dz, N, bias=bd, activation=Q.ACT_SILU_GATE,
                                cfg=Q.make_config(variant=5, split_k=split, tile_n=2)))
    assert rel_err(y, oracle.epilogue(oracle.gemm(x, q, z, s), b, act=1)) <= TOL
    say("kstream bias split=%d" % split)
    y = from_dev_y(Q.gemm_fused(xd, dw, ds, dz, N, bias=bd, cfg=Q.make_config(variant=5, split_k=split, tile_n=1)))
    assert rel_err(y, oracle.epilogue(oracle.gemm(x, q, z, s), b)) <= TOL
    # the gated form needs a gate tile and its up tile in one wave
    with pytest.raises(Q.QuickError):
        Q.gemm_fused(xd, dw, ds, dz, N, bias=bd, activation=Q.ACT_SILU_GATE,
                     cfg=Q.make_config(variant=5, split_k=split, tile_n=1))


def test_kstream_rejected_configs():
    K, N = 1024, 64
    x, q, z, s = rand_case(3, 17, K, N)
    p = Packed(q, z, s)
    xd = to_dev_x(x)
    bad = [(17, dict(variant=5)),                        # more than 16 rows
           (16, dict(variant=5, tile_n=4)),              # 1 or 2 n-tiles per wave
           (16, dict(variant=5, tile_m=16)),             # no row tile
           (16, dict(variant=5, split_k=K // 128 + 1))]  # more slices than k-groups
    for M, cfg in bad:
        say("rejected M=%d cfg=%s" % (M, cfg))
        with pytest.raises(Q.QuickError):
            p.gemm(xd[:M].contiguous(), cfg=Q.make_config(**cfg))
