"""Parity of the HIP GEMM (through the C ABI) with the CPU oracle.

* every kernel variant, tile and split on ragged shapes that span several
  tiles and a partial tail, element by element against the oracle;
* exact cases: one-hot activations give RNE_f16((q - z) * s) bit for bit;
  integer data give the integer GEMM bit for bit under any split order;
* metamorphic properties: doubling the scales doubles y exactly, permuting
  rows of x permutes rows of y exactly, permuting whole 16-column tiles of
  (q, z, s) permutes columns of y exactly; run-to-run determinism; guard
  rows around y stay untouched; caller workspace and non-default stream.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2402_10076_amd as Q
from gpu_util import TOL, Packed, f16_values, from_dev_y, rand_case, rel_err, run, say, to_dev_x

pytestmark = pytest.mark.gpu

STREAM_CFGS = [dict(variant=1, split_k=w, tile_n=p) for w in (1, 2, 4, 8) for p in (1, 2)]
TILES = ((16, 16), (16, 32), (32, 16), (32, 32), (64, 16), (64, 32), (128, 16), (128, 32))
TILED_CFGS = [dict(variant=2, tile_m=bm, tile_n=wn, split_k=s) for bm, wn in TILES for s in (1, 3)]
# stream-K: 8 and 24 resident workgroups split most tiles across workgroups;
# 0 = all resident workgroups (clamped to the work units)
STREAMK_CFGS = [dict(variant=3, tile_m=bm, tile_n=wn, split_k=g) for bm, wn in TILES for g in (8, 24, 0)]
# the tiled kernel on the 32x32x16 instruction (pairs of n-tiles, 32-row blocks)
TILES32 = ((32, 32), (64, 32), (128, 32))
TILED32_CFGS = ([dict(variant=6, tile_m=bm, tile_n=wn, split_k=s) for bm, wn in TILES32 for s in (1, 3)] +
                [dict(variant=7, tile_m=bm, tile_n=wn, split_k=g) for bm, wn in TILES32 for g in (8, 24, 0)])


def _check(M, K, N, cfg, seed):
    say("case M=%d K=%d N=%d cfg=%s" % (M, K, N, cfg))
    x, q, z, s = rand_case(seed, M, K, N)
    y = run(x, q, z, s, Q.make_config(**cfg) if cfg else None)
    ref = oracle.gemm(x, q, z, s)
    err = rel_err(y, ref)
    assert err <= TOL, "rel err %.3g for M=%d K=%d N=%d cfg=%s" % (err, M, K, N, cfg)
    return err


@pytest.mark.parametrize("cfg", STREAM_CFGS, ids=lambda c: "w%d_p%d" % (c["split_k"], c["tile_n"]))
@pytest.mark.parametrize("M", [1, 3, 16, 17, 33, 64])
def test_stream_variants(M, cfg):
    for K, N in ((384, 48), (1152, 80)):
        _check(M, K, N, cfg, seed=M * 1000 + K + N)


@pytest.mark.parametrize("waves,npw", [(1, 1), (1, 2), (4, 1), (4, 2)])
@pytest.mark.parametrize("M", [1, 3, 16])
def test_stream_ring_regimes(M, waves, npw):
    """Per-wave k-ranges on both sides of every register-ring depth the stream
    kernel uses (D = 4, 8, 16): a single pass (up to D units), one partial
    trip (D+1 .. 2D-1), and the peeled first trip plus the steady loop and a
    ragged tail (2D and more); activations staged in LDS (small M*K) or
    loaded from L2."""
    cfg = dict(variant=1, split_k=waves, tile_n=npw)
    for units in (3, 4, 5, 7, 8, 9, 15, 16, 17, 31, 32, 35, 69):
        _check(M, 128 * units * waves, 48, cfg, seed=units * 10 + M)


@pytest.mark.parametrize("cfg", TILED_CFGS, ids=lambda c: "bm%d_wn%d_s%d" % (c["tile_m"], c["tile_n"], c["split_k"]))
@pytest.mark.parametrize("M", [1, 65, 129, 300])
def test_tiled_variants(M, cfg):
    for K, N in ((384, 80), (640, 528)):
        _check(M, K, N, cfg, seed=M * 1000 + K + N + 7)


@pytest.mark.parametrize("cfg", TILED32_CFGS,
                         ids=lambda c: "v%d_bm%d_wn%d_s%d" % (c["variant"], c["tile_m"], c["tile_n"], c["split_k"]))
@pytest.mark.parametrize("M", [1, 33, 65, 129, 300])
def test_tiled32_variants(M, cfg):
    """Ragged shapes: N not a multiple of the 32-column pair (a lone last
    n-tile, clamped and never stored), M tails inside 32-row blocks, K slices
    and stream-K pieces across tiles."""
    for K, N in ((384, 80), (640, 528), (2304, 272)):
        _check(M, K, N, cfg, seed=M * 1000 + K + N + 17)


@pytest.mark.parametrize("cfg", STREAMK_CFGS, ids=lambda c: "bm%d_wn%d_g%d" % (c["tile_m"], c["tile_n"], c["split_k"]))
@pytest.mark.parametrize("M", [1, 65, 300])
def test_streamk_variants(M, cfg):
    for K, N in ((384, 80), (640, 528), (2304, 272)):
        _check(M, K, N, cfg, seed=M * 1000 + K + N + 11)


def test_kstream_deterministic_and_caller_workspace():
    """Slices summed in slice order: repeated calls give identical bits, with
    the internal or a caller workspace, whose counters are left zero."""
    M, K, N = 3, 8192, 528
    x, q, z, s = rand_case(77, M, K, N)
    p = Packed(q, z, s)
    xd = to_dev_x(x)
    cfg = Q.make_config(variant=5, split_k=5, tile_n=1)
    nb = Q.workspace_bytes(M, N, K, cfg)
    ws = torch.zeros(nb // 4 + 1, dtype=torch.int32, device="cuda")
    say("kstream determinism ws=%d" % nb)
    y0 = from_dev_y(p.gemm(xd, cfg=cfg))
    y1 = from_dev_y(p.gemm(xd, cfg=cfg, workspace=ws))
    y2 = from_dev_y(p.gemm(xd, cfg=cfg, workspace=ws))
    assert np.array_equal(y0, y1) and np.array_equal(y1, y2)
    assert int(ws[:Q.WS_COUNTER_BYTES // 4].abs().sum().item()) == 0
    assert rel_err(y0, oracle.gemm(x, q, z, s)) <= TOL


@pytest.mark.parametrize("G", [16, 32, 64])
def test_streamk_many_pieces_per_tile(G):
    """One output tile, 32 k-groups over G workgroups: every tile is summed
    from G / 1 .. pieces by the last arriving workgroup."""
    _check(16, 4096, 128, dict(variant=3, tile_m=16, tile_n=16, split_k=G), seed=G)
    _check(100, 4096, 256, dict(variant=3, tile_m=128, tile_n=32, split_k=G), seed=G + 1)


@pytest.mark.parametrize("rounds", [1.0, 2.0, 2.25, 2.5, 3.75])
@pytest.mark.parametrize("variant,wn", [(3, 16), (7, 32)])
def test_streamk_rounds_then_pieces(rounds, variant, wn):
    """Stream-K on 16 workgroups runs whole rounds of tiles one per workgroup,
    then splits the rest of the tiles: whole rounds only (1, 2), a quarter
    round merged into the last whole one (2.25), a half and three quarters
    of a round in pieces (2.5, 3.75)."""
    G, bm = 16, 32
    T = int(rounds * G)
    M = 4 * bm                      # 4 m-tiles per n-tile
    N = (T // 4) * 8 * wn           # T / 4 n-tiles of 8 waves x wn columns
    _check(M, 1024, N, dict(variant=variant, tile_m=bm, tile_n=wn, split_k=G), seed=int(rounds * 100) + variant)


@pytest.mark.parametrize("K,N", [(128, 16), (128, 272), (256, 16), (128, 4112)])
@pytest.mark.parametrize("M", [1, 17, 200])
def test_smallest_k_and_n(M, K, N):
    """One k-group and one n-tile, the edges of the tile space: every
    configuration that accepts the shape (stream, tiled and its split and
    stream-K schedules on both matrix instructions, sliced) matches the
    oracle element by element.  A split-K request above K / 128 slices is
    INVALID_ARG; stream-K on fewer than 8 tiles x k-groups runs whole
    tiles."""
    x, q, z, s = rand_case(M * 7 + K + N, M, K, N)
    p = Packed(q, z, s)
    xd = to_dev_x(x)
    ref = oracle.gemm(x, q, z, s)
    cfgs = [None] + [dict(variant=1, split_k=w, tile_n=n) for w in (1, 8) for n in (1, 2)] + \
        [dict(variant=v, tile_m=bm, tile_n=wn, split_k=sk) for v, sk in ((2, 1), (2, 2), (3, 0), (3, 8))
         for bm, wn in ((16, 16), (32, 32), (128, 32))] + \
        [dict(variant=v, tile_m=64, tile_n=32, split_k=sk) for v, sk in ((6, 1), (6, 2), (7, 0))] + \
        [dict(variant=5, split_k=0, tile_n=n) for n in (1, 2)]
    ran = 0
    for c in cfgs:
        if c and c["variant"] == 1 and M > 64:
            continue
        if c and c["variant"] == 5 and M > 16:
            continue
        if c and c["variant"] in (2, 6) and c["split_k"] > K // 128:
            with pytest.raises(Q.QuickError) as e:
                p.gemm(xd, cfg=Q.make_config(**c))
            assert e.value.status == Q.QUICK_ERR_INVALID_ARG
            continue
        say("smallest K=%d N=%d M=%d cfg=%s" % (K, N, M, c))
        y = from_dev_y(p.gemm(xd, cfg=Q.make_config(**c) if c else None))
        assert rel_err(y, ref) <= TOL, c
        ran += 1
    assert ran >= 12


@pytest.mark.parametrize("M", [1, 2, 5, 16, 31, 64, 65, 96, 127, 200, 513])
def test_auto_config_small_shapes(M):
    _check(M, 1024, 272, None, seed=M)


@pytest.mark.parametrize("M", [9, 16])
def test_auto_config_sliced_stream_shapes(M):
    """Shapes the automatic plan gives the sliced stream kernel (>= 128
    workgroups), and an explicit stream-kernel choice with its other fields
    left to the defaults."""
    assert Q.select_config(M, 8192, 4096)["variant"] == Q.VARIANT_KSTREAM
    _check(M, 4096, 8192, None, seed=40 + M)
    _check(M, 2048, 272, dict(variant=1), seed=50 + M)


def test_c1_toy_full_output():
    """16 x 512 x 512, group 128, full output against the oracle."""
    import workloads as W
    x, q, z, s = W.shape_inputs(W.C1, 0, 16)
    y = run(x, q, z, s)
    err = rel_err(y, oracle.gemm(x, q, z, s))
    say("C1 rel err %.3g" % err)
    assert err <= TOL


@pytest.mark.parametrize("cfg", [None, dict(variant=1, split_k=4, tile_n=2), dict(variant=2, tile_m=64, tile_n=32, split_k=2),
                                 dict(variant=2, tile_m=128, tile_n=32, split_k=1),
                                 dict(variant=5, split_k=3, tile_n=1), dict(variant=5, split_k=1, tile_n=2),
                                 dict(variant=6, tile_m=128, tile_n=32, split_k=1),
                                 dict(variant=6, tile_m=32, tile_n=32, split_k=2),
                                 dict(variant=7, tile_m=64, tile_n=32, split_k=16)])
def test_one_hot_rows_give_exact_dequant(cfg):
    """x row m = e_{k_m}: y[m][n] is a single product, so it must equal the
    binary16 rounding of (q - z) * s exactly."""
    K, N = 512, 96
    M = 16 if cfg is None or cfg["variant"] in (1, 5) else 100
    g = np.random.Generator(np.random.PCG64(5))
    _, q, z, s = rand_case(6, 1, K, N)
    ks = g.choice(K, size=M, replace=False)
    x = np.zeros((M, K), np.uint16)
    x[np.arange(M), ks] = 0x3C00
    y = run(x, q, z, s, Q.make_config(**cfg) if cfg else None)
    W = oracle.dequant(q, z, s)
    want = oracle.f64_to_f16(W[ks])
    assert np.array_equal(y, want), "dequantized value mismatch at %d entries" % int((y != want).sum())


KSTREAM_EXACT = [dict(variant=5, split_k=1, tile_n=2), dict(variant=5, split_k=5, tile_n=1)]


@pytest.mark.parametrize("cfg", [None] + STREAM_CFGS[::3] + TILED_CFGS[::3] + STREAMK_CFGS[::4] + KSTREAM_EXACT +
                         TILED32_CFGS[::2])
def test_integer_data_exact_under_any_split(cfg):
    """s = 1, z = 8, q in {7,8,9}, x in {-1,0,1}: every partial sum is a small
    integer, so any summation order is exact and y equals int64 x . (q - z)."""
    M = 48 if cfg is None or cfg["variant"] == 1 else 16 if cfg["variant"] == 5 else 150
    K, N = 1024, 80
    g = np.random.Generator(np.random.PCG64(9))
    xi = g.integers(-1, 2, (M, K))
    qi = g.integers(7, 10, (K, N))
    ref = xi @ (qi - 8)
    assert np.abs(ref).max() <= 2048
    x = xi.astype(np.float16).view(np.uint16)
    z = np.full((K // 128, N), 8, np.uint8)
    s = np.full((K // 128, N), 0x3C00, np.uint16)
    y = run(x, qi.astype(np.uint8), z, s, Q.make_config(**cfg) if cfg else None)
    assert np.array_equal(f16_values(y), ref.astype(np.float64))


@pytest.mark.parametrize("M,cfg", [(7, None), (64, None), (200, None), (16, dict(variant=5, split_k=3, tile_n=1)),
                                   (9, dict(variant=5, split_k=2, tile_n=2))],
                         ids=["7", "64", "200", "16_sliced", "9_sliced"])
def test_metamorphic_scale_rows_tiles(M, cfg):
    K, N = 768, 96
    cfg = Q.make_config(**cfg) if cfg else None
    x, q, z, s = rand_case(11 + M, M, K, N)
    p = Packed(q, z, s)
    xd = to_dev_x(x)
    y = from_dev_y(p.gemm(xd, cfg=cfg))
    # doubling the scales doubles y exactly (outside the binary16 subnormal band)
    s2 = (f16_values(s) * 2).astype(np.float16).view(np.uint16)
    y2 = run(x, q, z, s2, cfg)
    yv, y2v = f16_values(y), f16_values(y2)
    keep = np.abs(yv) >= 2.0 ** -14
    assert np.array_equal(y2v[keep], 2 * yv[keep])
    # permuting rows of x permutes rows of y
    perm = np.random.Generator(np.random.PCG64(M)).permutation(M)
    yp = from_dev_y(p.gemm(to_dev_x(x[perm]), cfg=cfg))
    assert np.array_equal(yp, y[perm])
    # permuting whole 16-column tiles of (q, z, s) permutes columns of y
    tperm = np.random.Generator(np.random.PCG64(M + 1)).permutation(N // 16)
    cols = (tperm[:, None] * 16 + np.arange(16)[None, :]).reshape(-1)
    yt = run(x, q[:, cols], z[:, cols], s[:, cols], cfg)
    assert np.array_equal(yt, y[:, cols])
    # determinism
    for _ in range(3):
        assert np.array_equal(from_dev_y(p.gemm(xd, cfg=cfg)), y)
    torch.cuda.synchronize()


@pytest.mark.parametrize("M", [5, 130])
def test_guard_rows_untouched(M):
    K, N = 512, 64
    x, q, z, s = rand_case(21, M, K, N)
    p = Packed(q, z, s)
    big = torch.full((M + 2, N), float("nan"), dtype=torch.float16, device="cuda")
    p.gemm(to_dev_x(x), y=big[1:M + 1])
    torch.cuda.synchronize()
    out = big.cpu()
    assert torch.isnan(out[0]).all() and torch.isnan(out[M + 1]).all()
    assert rel_err(from_dev_y(out[1:M + 1].contiguous()), oracle.gemm(x, q, z, s)) <= TOL


def test_caller_workspace_and_side_stream():
    M, K, N = 192, 1024, 256
    x, q, z, s = rand_case(31, M, K, N)
    p = Packed(q, z, s)
    xd = to_dev_x(x)
    cfg = Q.make_config(variant=2, tile_m=64, tile_n=32, split_k=4)
    y_int = from_dev_y(p.gemm(xd, cfg=cfg))
    need = Q.workspace_bytes(M, N, K, cfg)
    assert need > 0
    ws = torch.zeros(need // 4, dtype=torch.float32, device="cuda")  # arrival counters start at zero
    side = torch.cuda.Stream()
    with torch.cuda.stream(side):
        y_ws = p.gemm(xd, cfg=cfg, workspace=ws, stream=side)
    side.synchronize()
    assert np.array_equal(from_dev_y(y_ws), y_int)
    small = torch.empty(need // 8, dtype=torch.float32, device="cuda")
    with pytest.raises(Q.QuickError):
        p.gemm(xd, cfg=cfg, workspace=small)


def test_streamk_caller_workspace_reuse_and_determinism():
    M, K, N = 300, 2304, 528
    x, q, z, s = rand_case(41, M, K, N)
    p = Packed(q, z, s)
    xd = to_dev_x(x)
    cfg = Q.make_config(variant=3, tile_m=64, tile_n=32, split_k=24)
    need = Q.workspace_bytes(M, N, K, cfg)
    assert need > Q.WS_COUNTER_BYTES
    ws = torch.zeros(need // 4, dtype=torch.float32, device="cuda")  # counters start at zero
    y0 = from_dev_y(p.gemm(xd, cfg=cfg, workspace=ws))
    assert rel_err(y0, oracle.gemm(x, q, z, s)) <= TOL
    torch.cuda.synchronize()
    # every call leaves the counters at zero, and the fixed k-order sum makes
    # repeated calls bit-identical
    assert int(torch.count_nonzero(ws[:Q.WS_COUNTER_BYTES // 4])) == 0
    for _ in range(3):
        assert np.array_equal(from_dev_y(p.gemm(xd, cfg=cfg, workspace=ws)), y0)
    assert int(torch.count_nonzero(ws[:Q.WS_COUNTER_BYTES // 4])) == 0
    # the same through the library-owned workspace, interleaved with split-K
    # calls that share it
    sk2 = Q.make_config(variant=2, tile_m=64, tile_n=32, split_k=3)
    for _ in range(2):
        assert np.array_equal(from_dev_y(p.gemm(xd, cfg=cfg)), y0)
        assert rel_err(from_dev_y(p.gemm(xd, cfg=sk2)), f16_values(y0)) <= TOL


def test_m_zero_is_noop():
    K, N = 256, 32
    _, q, z, s = rand_case(1, 1, K, N)
    p = Packed(q, z, s)
    y = p.gemm(torch.empty((0, K), dtype=torch.float16, device="cuda"))
    assert tuple(y.shape) == (0, N)
    # every explicit kernel choice
    K = 2048
    _, q, z, s = rand_case(2, 1, K, N)
    p = Packed(q, z, s)
    for cfg in (dict(variant=1), dict(variant=5, split_k=2), dict(variant=3, tile_m=16, tile_n=16),
                dict(variant=2, tile_m=128, tile_n=32, split_k=2)):
        y = p.gemm(torch.empty((0, K), dtype=torch.float16, device="cuda"), cfg=Q.make_config(**cfg))
        assert tuple(y.shape) == (0, N)
    torch.cuda.synchronize()
