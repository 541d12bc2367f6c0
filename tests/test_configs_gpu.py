"""The five workload configurations at full size, on the launch
configurations the benchmark times (the built-in rules, and for the
Llama-2-7B / 70B sets also the tune table bench.py loads).

Against the oracle, per (shape, M) point: every row, and one column of every
16-column n-tile (the position inside the tile rotating with the tile index,
so all 16 positions occur) plus the first and last 256 columns.  Every
output tile of every schedule -- stream-K pieces, split-K slices, the sliced
kernel's slices, the grouped form's remainder launch -- therefore has
outputs checked against the oracle.  Rows of x are drawn in order, so the
oracle runs once per shape at the largest M and each smaller M compares
against its leading rows.

Beside it, as a secondary full-coverage check (not the oracle): every output
element against an fp32 GEMM through torch on a torch-dequantized W (plain
elementwise ops and a matmul, independent of the HIP kernels).  Inputs come
from workloads.py with the configurations' seeds and distributions."""
import os

import numpy as np
import pytest
import torch

import oracle
import paper_2402_10076_amd as Q
import workloads as W
from gpu_util import TOL, Packed, from_dev_y, rel_err, say, to_dev_x

pytestmark = pytest.mark.gpu


def tile_columns(N: int) -> np.ndarray:
    """Column 16t + (t mod 16) of every n-tile t, and the first and last 256 columns."""
    t = np.arange(N // 16)
    cols = np.concatenate([16 * t + (t % 16), np.arange(min(256, N)), np.arange(max(0, N - 256), N)])
    return np.unique(cols).astype(np.int64)


class TorchReference:
    """y = x . W in fp32 through torch, W dequantized by torch elementwise
    ops on the device: the secondary check over every output element."""

    def __init__(self, q, z, s):
        dev = "cuda"
        g = q.shape[0] // z.shape[0]
        qd = torch.from_numpy(q).to(dev).float()
        zd = torch.from_numpy(z).to(dev).float().repeat_interleave(g, 0)
        sd = torch.from_numpy(s.view(np.float16)).to(dev).float().repeat_interleave(g, 0)
        self.W = (qd - zd) * sd          # exact: |q - z| <= 15 times a binary16 value
        del qd, zd, sd

    def err(self, x_dev, y_bits) -> float:
        prev = torch.backends.cuda.matmul.allow_tf32
        torch.backends.cuda.matmul.allow_tf32 = False
        try:
            ref = (x_dev.float() @ self.W).double().cpu().numpy()
        finally:
            torch.backends.cuda.matmul.allow_tf32 = prev
        return rel_err(y_bits, ref)


_ORACLE = {}


def oracle_rows(key, x_all, q, z, s, cols):
    """Oracle output for all rows of x_all over `cols`, computed once per
    (config, shape) key and kept while the tests stay on that config."""
    if key not in _ORACLE:
        for k in [k for k in _ORACLE if k[0] != key[0]]:
            del _ORACLE[k]
        _ORACLE[key] = oracle.gemm(x_all, q, z, s, cols=cols)
    return _ORACLE[key]


def _check_point(tag, p, x_dev, y_ref_rows, cols, tref, M):
    y = from_dev_y(p.gemm(x_dev))
    assert y.shape == (M, p.N)
    err = rel_err(y[:, cols], y_ref_rows[:M])
    err32 = tref.err(x_dev, y)
    say("%s M=%d rel_err=%.3g (%d rows x %d columns), all outputs vs fp32 torch %.3g" % (
        tag, M, err, M, len(cols), err32))
    assert err <= TOL, "%s M=%d: rel err %.3g" % (tag, M, err)
    assert err32 <= TOL, "%s M=%d: rel err %.3g against the fp32 GEMM" % (tag, M, err32)


TUNE_TABLE = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "paper_2402_10076_amd",
                          "tune_mi355x.txt")


@pytest.fixture
def bench_plans(request):
    """The plans bench.py launches: the library's MI355X tune table for the
    Llama-2-7B / 70B shapes (the built-in rules for everything else)."""
    if request.param == "tuned":
        Q.tune_table_load(TUNE_TABLE)
    yield request.param
    Q.tune_table_clear()


@pytest.mark.parametrize("cid,bench_plans", [(2, "rules"), (2, "tuned"), (3, "rules"), (5, "rules"), (5, "tuned")],
                         indirect=["bench_plans"])
def test_llama_config(cid, bench_plans):
    cfg = W.CONFIGS[cid]
    for si, sh in enumerate(cfg.shapes):
        say("C%d %s K=%d N=%d: generating" % (cid, sh.name, sh.K, sh.N))
        x_all = W.draw_x(cid, si, max(sh.Ms), sh.K, cfg.outliers)
        q, z, s = W.draw_weights(cid, si, sh.K, sh.N)
        cols = tile_columns(sh.N)
        ref = oracle_rows((cid, si), x_all, q, z, s, cols)
        p = Packed(q, z, s)
        tref = TorchReference(q, z, s)
        xd_all = to_dev_x(x_all)
        for M in sh.Ms:
            _check_point("C%d %s %s" % (cid, bench_plans, sh.name), p, xd_all[:M], ref, cols, tref, M)
        del p, tref, xd_all
        torch.cuda.empty_cache()


def test_mixtral_experts():
    routes = W.mixtral_routing()
    assert sum(len(r) for r in routes) == W.MIXTRAL_TOKENS * W.MIXTRAL_TOPK
    xt = W.mixtral_tokens()
    for e in range(W.MIXTRAL_EXPERTS):
        Me = len(routes[e])
        for which, name in enumerate(("w1", "w3", "w2")):
            q, z, s = W.mixtral_expert_weights(e, which)
            x = xt[routes[e]] if which < 2 else W.mixtral_w2_input(e, Me)
            cols = tile_columns(q.shape[1])
            ref = oracle.gemm(x, q, z, s, cols=cols)
            _check_point("C4 expert%d %s" % (e, name), Packed(q, z, s), to_dev_x(x), ref, cols,
                         TorchReference(q, z, s), Me)


def test_mixtral_grouped():
    """The same expert GEMMs as one grouped call per weight (w1, w3 over the
    routed tokens, gathered in the kernel; w2 over the experts' stacked
    inputs), each expert's block of rows against the oracle on every row
    and the n-tile columns, and every output against fp32 torch."""
    routes = W.mixtral_routing()
    xt = W.mixtral_tokens()
    counts = [len(r) for r in routes]
    offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    rows = np.concatenate(routes).astype(np.int32)
    od = torch.from_numpy(offsets).cuda()
    rd = torch.from_numpy(rows).cuda()
    for which, name in enumerate(("w1", "w3", "w2")):
        experts = [W.mixtral_expert_weights(e, which) for e in range(W.MIXTRAL_EXPERTS)]
        K, N = experts[0][0].shape
        dw, ds, dz = Q.to_device(*Q.pack_experts(experts))
        if which < 2:
            x = xt
            y = from_dev_y(Q.grouped_gemm(to_dev_x(xt), od, dw, ds, dz, N, rows=rd))
        else:
            x = np.concatenate([W.mixtral_w2_input(e, counts[e]) for e in range(W.MIXTRAL_EXPERTS)])
            y = from_dev_y(Q.grouped_gemm(to_dev_x(x), od, dw, ds, dz, N))
        cols = tile_columns(N)
        for e in range(W.MIXTRAL_EXPERTS):
            lo, hi = offsets[e], offsets[e + 1]
            xr = x[rows[lo:hi]] if which < 2 else x[lo:hi]
            ref = oracle.gemm(xr, *experts[e], cols=cols)
            err = rel_err(y[lo:hi][:, cols], ref)
            err32 = TorchReference(*experts[e]).err(to_dev_x(xr), y[lo:hi])
            say("C4 grouped %s expert%d M=%d rel_err=%.3g, all outputs vs fp32 torch %.3g" % (
                name, e, counts[e], err, err32))
            assert err <= TOL and err32 <= TOL
        del dw, ds, dz
        torch.cuda.empty_cache()


def test_tile_columns_cover_every_tile_and_position():
    cols = tile_columns(57344)
    assert set(np.unique(cols // 16)) == set(range(57344 // 16))
    assert set(np.unique(cols % 16)) == set(range(16))
    assert cols[0] == 0 and cols[-1] == 57343 and np.all(np.diff(cols) > 0)
    assert len(tile_columns(512)) == 512
