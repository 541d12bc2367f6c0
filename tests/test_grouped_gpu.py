"""Grouped (mixture-of-experts) GEMM on the GPU through the C ABI
(include/quick_grouped.h) against the oracle's grouped form, plus bit-exact
agreement with the dense GEMM applied expert by expert."""
import numpy as np
import pytest
import torch

import oracle
import paper_2402_10076_amd as Q
from gpu_util import TOL, Packed, from_dev_y, rand_case, rel_err, say, to_dev_x

pytestmark = pytest.mark.gpu


def _experts(seed, E, K, N):
    g = np.random.Generator(np.random.PCG64(seed))
    out = []
    for _ in range(E):
        q = g.integers(0, 16, (K, N), dtype=np.uint8)
        z = g.integers(0, 16, (K // 128, N), dtype=np.uint8)
        s = g.uniform(0.002, 0.02, (K // 128, N)).astype(np.float16).view(np.uint16)
        out.append((q, z, s))
    return out


def _routing(seed, T, E, counts=None, topk=2):
    """Top-k routing of T tokens (or explicit per-expert row counts with
    random tokens): (rows, offsets) with each expert's rows in token order."""
    g = np.random.Generator(np.random.PCG64(seed))
    if counts is None:
        picks = np.stack([g.choice(E, size=topk, replace=False) for _ in range(T)])
        per = [np.nonzero((picks == e).any(axis=1))[0] for e in range(E)]
    else:
        per = [np.sort(g.integers(0, T, c)) for c in counts]
    offsets = np.concatenate([[0], np.cumsum([len(p) for p in per])]).astype(np.int32)
    rows = np.concatenate(per).astype(np.int32) if offsets[-1] else np.zeros(0, np.int32)
    return rows, offsets


class Grouped:
    def __init__(self, experts):
        self.E = len(experts)
        self.K, self.N = experts[0][0].shape
        self.dw, self.ds, self.dz = Q.to_device(*Q.pack_experts(experts))

    def run(self, x_dev, rows, offsets, cfg=None, R=None, y=None, workspace=None):
        r = torch.from_numpy(rows).cuda() if rows is not None else None
        o = torch.from_numpy(offsets).cuda()
        return Q.grouped_gemm(x_dev, o, self.dw, self.ds, self.dz, self.N, rows=r, R=R, y=y, cfg=cfg,
                              workspace=workspace)


CFGS = [None,
        dict(variant=2, split_k=1, tile_m=16, tile_n=16),
        dict(variant=2, split_k=3, tile_m=32, tile_n=16),
        dict(variant=2, split_k=1, tile_m=64, tile_n=32),
        dict(variant=2, split_k=2, tile_m=128, tile_n=32),
        dict(variant=3, split_k=8, tile_m=16, tile_n=16),
        dict(variant=3, split_k=64, tile_m=32, tile_n=16),
        dict(variant=3, split_k=0, tile_m=64, tile_n=32),
        dict(variant=3, split_k=16, tile_m=128, tile_n=32)]


@pytest.mark.parametrize("cfg", CFGS, ids=lambda c: "auto" if c is None else
                         "v%d_s%d_%dx%d" % (c["variant"], c["split_k"], c["tile_m"], c["tile_n"]))
def test_grouped_against_oracle(cfg):
    """5 experts with uneven rows (one empty, one with a ragged 1-row tail),
    gathered tokens with repeats; every output element against the oracle."""
    T, K, N = 90, 384, 272
    E = 5
    experts = _experts(7, E, K, N)
    x, _, _, _ = rand_case(8, T, K, 16)
    rows, offsets = _routing(9, T, E, counts=[37, 0, 129, 1, 66])
    G = Grouped(experts)
    say("grouped cfg=%s R=%d" % (cfg, offsets[-1]))
    y = from_dev_y(G.run(to_dev_x(x), rows, offsets, cfg=Q.make_config(**cfg) if cfg else None))
    ref = oracle.grouped_gemm(x, rows, offsets, experts)
    err = rel_err(y, ref)
    say("  rel_err=%.3g" % err)
    assert err <= TOL


@pytest.mark.parametrize("tile", [(16, 16), (32, 16), (64, 32), (128, 32)])
def test_grouped_equals_dense_per_expert_bitwise(tile):
    """Data-parallel grouped tiles compute the same sums in the same order as
    the dense GEMM on each expert's gathered rows: identical bits."""
    T, K, N = 200, 512, 512
    E = 4
    experts = _experts(11, E, K, N)
    x, _, _, _ = rand_case(12, T, K, 16)
    rows, offsets = _routing(13, T, E)
    cfg = dict(variant=2, split_k=1, tile_m=tile[0], tile_n=tile[1])
    say("grouped vs dense tile=%s R=%d" % (tile, offsets[-1]))
    y = from_dev_y(Grouped(experts).run(to_dev_x(x), rows, offsets, cfg=Q.make_config(**cfg)))
    for e in range(E):
        lo, hi = offsets[e], offsets[e + 1]
        p = Packed(*experts[e])
        ye = from_dev_y(p.gemm(to_dev_x(x[rows[lo:hi]]), cfg=Q.make_config(**cfg)))
        assert np.array_equal(y[lo:hi], ye), "expert %d differs from the dense GEMM" % e


def test_grouped_identity_rows_single_expert_equals_dense():
    """rows = NULL and one expert: the plain GEMM (same data-parallel tile)."""
    M, K, N = 77, 640, 528
    x, q, z, s = rand_case(21, M, K, N)
    offsets = np.array([0, M], np.int32)
    cfg = Q.make_config(variant=2, split_k=1, tile_m=32, tile_n=16)
    say("grouped identity rows M=%d" % M)
    y = from_dev_y(Grouped([(q, z, s)]).run(to_dev_x(x), None, offsets, cfg=cfg))
    yd = from_dev_y(Packed(q, z, s).gemm(to_dev_x(x), cfg=cfg))
    assert np.array_equal(y, yd)


def test_grouped_all_rows_one_expert_and_empty_edges():
    """Empty experts first and last, every row on one expert in the middle."""
    T, K, N = 48, 256, 256
    E = 6
    experts = _experts(31, E, K, N)
    x, _, _, _ = rand_case(32, T, K, 16)
    rows, offsets = _routing(33, T, E, counts=[0, 0, 0, 130, 0, 0])
    say("grouped one busy expert")
    for cfg in (None, Q.make_config(variant=2, split_k=2, tile_m=64, tile_n=32)):
        y = from_dev_y(Grouped(experts).run(to_dev_x(x), rows, offsets, cfg=cfg))
        assert rel_err(y, oracle.grouped_gemm(x, rows, offsets, experts)) <= TOL


def test_grouped_streamk_deterministic_and_caller_workspace():
    """Stream-K pieces are summed in k order: repeated calls, with the
    internal or a caller workspace, give identical bits; the workspace's
    counters are left zero."""
    T, K, N = 300, 2048, 512
    E = 8
    experts = _experts(41, E, K, N)
    x, _, _, _ = rand_case(42, T, K, 16)
    rows, offsets = _routing(43, T, E)
    G = Grouped(experts)
    xd = to_dev_x(x)
    cfg = Q.make_config(variant=3, split_k=40 * 8, tile_m=64, tile_n=32)
    R = int(offsets[-1])
    nb = Q.grouped_workspace_bytes(R, E, N, K, cfg)
    ws = torch.zeros(nb // 4 + 1, dtype=torch.int32, device="cuda")
    say("grouped stream-K determinism R=%d ws=%d" % (R, nb))
    y0 = from_dev_y(G.run(xd, rows, offsets, cfg=cfg))
    y1 = from_dev_y(G.run(xd, rows, offsets, cfg=cfg, workspace=ws))
    y2 = from_dev_y(G.run(xd, rows, offsets, cfg=cfg, workspace=ws))
    assert np.array_equal(y0, y1) and np.array_equal(y1, y2)
    assert int(ws[:Q.WS_COUNTER_BYTES // 4].abs().sum().item()) == 0
    assert rel_err(y0, oracle.grouped_gemm(x, rows, offsets, experts)) <= TOL


@pytest.mark.parametrize("counts", [[130, 149, 111, 20, 257, 0, 128, 200], [129, 131, 127, 128]])
def test_grouped_auto_full_height_two_parts(counts):
    """The automatic plan for about 128 rows per expert runs as two launches
    (128-row tiles over whole tiles and remainders of >= 64 rows, then 32-row
    tiles over the short remainders): every row against the oracle, the
    workspace query covering both launches, repeated calls identical."""
    T, K, N = 400, 512, 256
    E = len(counts)
    experts = _experts(81, E, K, N)
    x, _, _, _ = rand_case(82, T, K, 16)
    rows, offsets = _routing(83, T, E, counts=counts)
    R = int(offsets[-1])
    assert Q.grouped_select_config(R, E, N, K)["tile_m"] == 128
    G = Grouped(experts)
    xd = to_dev_x(x)
    say("grouped two parts R=%d counts=%s" % (R, counts))
    y0 = from_dev_y(G.run(xd, rows, offsets))
    nb = Q.grouped_workspace_bytes(R, E, N, K)
    ws = torch.zeros(nb // 4 + 1, dtype=torch.int32, device="cuda")
    y1 = from_dev_y(G.run(xd, rows, offsets, workspace=ws))
    assert np.array_equal(y0, y1)
    assert int(ws[:Q.WS_COUNTER_BYTES // 4].abs().sum().item()) == 0
    assert rel_err(y0, oracle.grouped_gemm(x, rows, offsets, experts)) <= TOL


def test_grouped_zero_rows_is_noop():
    experts = _experts(51, 2, 128, 16)
    G = Grouped(experts)
    x = torch.zeros((4, 128), dtype=torch.float16, device="cuda")
    y = G.run(x, np.zeros(0, np.int32), np.zeros(3, np.int32), R=0)
    torch.cuda.synchronize()
    assert y.shape == (0, 16)
