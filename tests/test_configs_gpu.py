"""The five workload configurations at full size, on the launch
configurations the benchmark times (the built-in rules, and for the
Llama-2-7B / 70B sets also the tune table bench.py loads), against the
oracle on sampled outputs: all rows up to 64 (else 64 sampled rows) and 256
sampled columns (the first 64, the last 64 and 128 random ones), every
(shape, M) point.  Inputs come from workloads.py with the configurations'
seeds and distributions."""
import os

import numpy as np
import pytest
import torch

import oracle
import paper_2402_10076_amd as Q
import workloads as W
from gpu_util import TOL, Packed, from_dev_y, rel_err, say, to_dev_x

pytestmark = pytest.mark.gpu


def _check_point(tag, p, x, q, z, s, M):
    xd = to_dev_x(x)
    y = from_dev_y(p.gemm(xd))
    rows = W.sample_rows(M)
    cols = W.sample_columns(p.N, 256)
    ref = oracle.gemm(x[rows], q, z, s, cols=cols)
    err = rel_err(y[np.ix_(rows, cols)], ref)
    say("%s M=%d rel_err=%.3g" % (tag, M, err))
    assert err <= TOL, "%s M=%d: rel err %.3g" % (tag, M, err)


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
        p = Packed(q, z, s)
        for M in sh.Ms:
            _check_point("C%d %s %s" % (cid, bench_plans, sh.name), p, x_all[:M], q, z, s, M)
        del p
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
            _check_point("C4 expert%d %s" % (e, name), Packed(q, z, s), x, q, z, s, Me)


def test_mixtral_grouped():
    """The same expert GEMMs as one grouped launch per weight (w1, w3 over
    the routed tokens, gathered in the kernel; w2 over the experts' stacked
    inputs), each expert's block against the oracle on sampled outputs."""
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
        cols = W.sample_columns(N, 256)
        for e in range(W.MIXTRAL_EXPERTS):
            lo = offsets[e]
            sub = W.sample_rows(counts[e])
            xr = x[rows[lo + sub]] if which < 2 else x[lo + sub]
            ref = oracle.gemm(xr, *experts[e], cols=cols)
            err = rel_err(y[np.ix_(lo + sub, cols)], ref)
            say("C4 grouped %s expert%d M=%d rel_err=%.3g" % (name, e, counts[e], err))
            assert err <= TOL
        del dw, ds, dz
        torch.cuda.empty_cache()
