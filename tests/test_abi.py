"""The C ABI without a GPU: the library loads, exports every function that
include/*.h declare, the headers compile as plain C, and every
validation path returns its status before touching the device."""
import ctypes
import os
import re
import subprocess
import tempfile

import numpy as np
import pytest

import paper_2402_10076_amd as Q

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = [os.path.join(ROOT, "include", h) for h in sorted(os.listdir(os.path.join(ROOT, "include")))
           if h.endswith(".h")]


def declared_functions():
    names = set()
    for h in HEADERS:
        src = re.sub(r"/\*.*?\*/", "", open(h).read(), flags=re.S)
        names |= set(re.findall(r"\b(quick_[a-z0-9_]+)\s*\(", src))
    return sorted(names)


def test_every_declared_symbol_is_exported():
    names = declared_functions()
    assert "quick_w4a16_gemm" in names and "quick_pack_weights" in names
    L = Q.lib()
    for n in names:
        assert hasattr(L, n), "libquick.so does not export %s" % n
    assert set(names) == set(Q.EXPORTED)


def test_header_is_plain_c_and_links():
    prog = r'''
#include "quick.h"
#include "quick_ablation.h"
#include "quick_fused.h"
#include "quick_grouped.h"
#include <stdio.h>
#include <string.h>
int main(void) {
    size_t a, b, c;
    if (quick_pack_format_version() != 1) return 1;
    if (quick_packed_sizes(256, 32, 128, &a, &b, &c) != QUICK_OK) return 2;
    if (a != 4096 || b != 32 || c != 128) return 3;
    if (quick_packed_sizes(256, 32, 64, &a, &b, &c) != QUICK_ERR_UNSUPPORTED) return 4;
    quick_config_t cfg;
    memset(&cfg, 0, sizeof cfg);
    if (quick_select_config(1, 4096, 4096, &cfg) != QUICK_OK || cfg.variant != 1) return 5;
    if (quick_w4a16_gemm(0, 0, 0, 0, 0, 0, 4096, 4096, 128, 0) != QUICK_OK) return 6;
    if (quick_ablation_gemm(0, 0, 0, 0, 0, 4, 4096, 4096, 3, 0) != QUICK_ERR_INVALID_ARG) return 7;
    if (quick_w4a16_grouped_gemm(0, 0, 0, 0, 0, 0, 0, 16, 0, 8, 4096, 4096, 128, 0) != QUICK_OK) return 8;
    if (QUICK_MAX_EXPERTS != 512) return 9;
    quick_epilogue_t e = {0, QUICK_ACT_SILU_GATE};
    if (quick_w4a16_gemm_fused(0, 0, 0, 0, 0, 0, 4096, 4096, 128, 0, &e, 0, 0, 0) != QUICK_OK) return 10;
    printf("%s\n", quick_status_string(QUICK_ERR_SHAPE));
    return 0;
}
'''
    with tempfile.TemporaryDirectory() as d:
        c = os.path.join(d, "t.c")
        exe = os.path.join(d, "t")
        open(c, "w").write(prog)
        libdir = os.path.dirname(Q.LIB_PATH)
        subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror", "-I", os.path.join(ROOT, "include"), c,
                        "-o", exe, os.path.join(libdir, "libquick.so"),
                        "-Wl,-rpath," + libdir], check=True)
        r = subprocess.run([exe], capture_output=True, text=True)
        assert r.returncode == 0, r.stdout + r.stderr
        assert "QUICK_ERR_SHAPE" in r.stdout


def _gemm(x, pw, ps, pz, y, M, N, K, group=128):
    return Q.lib().quick_w4a16_gemm(x, pw, ps, pz, y, M, N, K, group, None)


def test_gemm_validation_without_device():
    A = 0x10000  # fake, 256-byte aligned addresses: never dereferenced
    ok = dict(x=A, pw=A, ps=A, pz=A, y=A)
    assert _gemm(**ok, M=0, N=4096, K=4096) == Q.QUICK_OK
    assert _gemm(0, 0, 0, 0, 0, 0, 4096, 4096) == Q.QUICK_OK
    assert _gemm(**ok, M=-1, N=4096, K=4096) == Q.QUICK_ERR_SHAPE
    assert _gemm(**ok, M=4, N=4096, K=4000) == Q.QUICK_ERR_SHAPE
    assert _gemm(**ok, M=4, N=4088, K=4096) == Q.QUICK_ERR_SHAPE
    assert _gemm(**ok, M=4, N=0, K=4096) == Q.QUICK_ERR_SHAPE
    assert _gemm(**ok, M=4, N=4096, K=4096, group=64) == Q.QUICK_ERR_UNSUPPORTED
    assert _gemm(0, A, A, A, A, 4, 4096, 4096) == Q.QUICK_ERR_INVALID_ARG
    assert _gemm(A, A, A, A, 0, 4, 4096, 4096) == Q.QUICK_ERR_INVALID_ARG
    assert _gemm(A + 8, A, A, A, A, 4, 4096, 4096) == Q.QUICK_ERR_ALIGNMENT
    assert _gemm(A, A + 4, A, A, A, 4, 4096, 4096) == Q.QUICK_ERR_ALIGNMENT
    assert _gemm(A, A, A + 1, A, A, 4, 4096, 4096) == Q.QUICK_ERR_ALIGNMENT
    assert _gemm(A, A, A, A + 2, A, 4, 4096, 4096) == Q.QUICK_ERR_ALIGNMENT
    assert _gemm(A, A, A, A, A + 4, 4, 4096, 4096) == Q.QUICK_ERR_ALIGNMENT
    # 32-bit index limits: each at its first rejected value (the largest
    # accepted ones run on the GPU in test_limits_gpu.py)
    assert _gemm(**ok, M=4, N=1 << 20, K=1 << 17) == Q.QUICK_ERR_SHAPE
    assert _gemm(**ok, M=4, N=131072, K=65536) == Q.QUICK_ERR_SHAPE          # K*N/2 == 2^32 bytes
    assert _gemm(**ok, M=1 << 19, N=48, K=4096) == Q.QUICK_ERR_SHAPE         # M*K == 2^31
    assert _gemm(**ok, M=1 << 16, N=32768, K=128) == Q.QUICK_ERR_SHAPE       # M*N == 2^31
    assert _gemm(**ok, M=(1 << 24) + 1, N=16, K=128) == Q.QUICK_ERR_SHAPE    # M > 2^24


def test_noalloc_validation_without_device(tmp_path):
    """The allocation-free entry point reports argument errors, and a plan
    larger than its fixed scratch array, before any device work."""
    A = 0x10000
    L = Q.lib()

    def na(x=A, pw=A, ps=A, pz=A, y=A, M=4, N=4096, K=4096, group=128):
        return L.quick_w4a16_gemm_noalloc(x, pw, ps, pz, y, M, N, K, group, None)
    assert na(M=0) == Q.QUICK_OK
    assert na(M=-1) == Q.QUICK_ERR_SHAPE
    assert na(K=4000) == Q.QUICK_ERR_SHAPE
    assert na(group=64) == Q.QUICK_ERR_UNSUPPORTED
    assert na(x=0) == Q.QUICK_ERR_INVALID_ARG
    assert na(y=A + 4) == Q.QUICK_ERR_ALIGNMENT
    # every automatic plan of the benchmark shapes fits the scratch array
    for M, N, K in ((1024, 10240, 8192), (512, 57344, 8192), (128, 8192, 28672), (16, 12288, 4096)):
        assert 0 <= Q.workspace_bytes(M, N, K) <= Q.SCRATCH_BYTES
    # a tuned plan whose partial sums exceed it is refused
    big = tmp_path / "big.txt"
    big.write_text("quick-tune 1\n1024 57344 8192 2 8 128 32\n")
    Q.tune_table_load(str(big))
    try:
        assert Q.workspace_bytes(1024, 57344, 8192) > Q.SCRATCH_BYTES
        assert na(M=1024, N=57344, K=8192) == Q.QUICK_ERR_WORKSPACE
    finally:
        Q.tune_table_clear()


def test_gemm_ex_validation_without_device():
    A = 0x10000
    L = Q.lib()
    def ex(cfg, M=4, N=4096, K=4096, ws=None, wsb=0):
        return L.quick_w4a16_gemm_ex(A, A, A, A, A, M, N, K, 128, None, ctypes.byref(cfg), ws, wsb)
    assert ex(Q.make_config(variant=8)) == Q.QUICK_ERR_INVALID_ARG
    # the 32x32x16 tiled form: 32-column waves over 32, 64 or 128 rows
    assert ex(Q.make_config(variant=6, tile_m=64, tile_n=16)) == Q.QUICK_ERR_INVALID_ARG
    assert ex(Q.make_config(variant=6, tile_m=64, tile_n=64)) == Q.QUICK_ERR_INVALID_ARG
    assert ex(Q.make_config(variant=7, tile_m=16, tile_n=32)) == Q.QUICK_ERR_INVALID_ARG
    assert ex(Q.make_config(variant=7, tile_m=128, split_k=12)) == Q.QUICK_ERR_INVALID_ARG
    assert ex(Q.make_config(variant=6, split_k=33)) == Q.QUICK_ERR_INVALID_ARG
    assert Q.workspace_bytes(256, 4096, 4096, Q.make_config(variant=6, tile_m=128, tile_n=32, split_k=4)) == \
        Q.WS_COUNTER_BYTES + 4 * 256 * 4096 * 4
    assert Q.workspace_bytes(256, 4096, 4096, Q.make_config(variant=7, tile_m=128, tile_n=32, split_k=64)) == \
        Q.WS_COUNTER_BYTES + 2 * 64 * 128 * 256 * 4
    assert ex(Q.make_config(variant=5), M=17) == Q.QUICK_ERR_INVALID_ARG       # more than 16 rows
    assert ex(Q.make_config(variant=5, tile_n=3)) == Q.QUICK_ERR_INVALID_ARG
    assert ex(Q.make_config(variant=5, tile_m=16)) == Q.QUICK_ERR_INVALID_ARG
    assert ex(Q.make_config(variant=5, split_k=33)) == Q.QUICK_ERR_INVALID_ARG  # more slices than k-groups
    assert ex(Q.make_config(variant=5), M=1, N=16 * 8 * 4097, K=128) == Q.QUICK_ERR_INVALID_ARG  # counters
    assert ex(Q.make_config(variant=4), M=1) == Q.QUICK_ERR_INVALID_ARG       # reserved number
    assert ex(Q.make_config(variant=4), M=0) == Q.QUICK_ERR_INVALID_ARG
    assert ex(Q.make_config(variant=3, split_k=12)) == Q.QUICK_ERR_INVALID_ARG   # not a multiple of 8
    assert ex(Q.make_config(variant=3, split_k=8192)) == Q.QUICK_ERR_INVALID_ARG
    assert ex(Q.make_config(variant=3, tile_m=128, tile_n=64)) == Q.QUICK_ERR_INVALID_ARG
    assert ex(Q.make_config(variant=1), M=65) == Q.QUICK_ERR_INVALID_ARG
    assert ex(Q.make_config(variant=1, split_k=3)) == Q.QUICK_ERR_INVALID_ARG
    assert ex(Q.make_config(variant=1, tile_n=3)) == Q.QUICK_ERR_INVALID_ARG
    assert ex(Q.make_config(variant=2, tile_m=96)) == Q.QUICK_ERR_INVALID_ARG
    assert ex(Q.make_config(variant=2, tile_m=16, tile_n=64)) == Q.QUICK_ERR_INVALID_ARG
    assert ex(Q.make_config(variant=2, tile_n=48)) == Q.QUICK_ERR_INVALID_ARG
    assert ex(Q.make_config(variant=2, split_k=33)) == Q.QUICK_ERR_INVALID_ARG
    assert ex(Q.make_config(variant=2, tile_m=256, tile_n=64)) == Q.QUICK_ERR_INVALID_ARG
    assert ex(Q.make_config(variant=2, tile_m=128, tile_n=64)) == Q.QUICK_ERR_INVALID_ARG
    assert ex(Q.make_config(variant=2, tile_m=64, tile_n=64)) == Q.QUICK_ERR_INVALID_ARG   # withdrawn: it spilled
    cfg = Q.make_config(variant=2, tile_m=128, tile_n=32, split_k=4)
    need = Q.workspace_bytes(256, 4096, 4096, cfg)
    assert need == Q.WS_COUNTER_BYTES + 4 * 256 * 4096 * 4
    assert ex(cfg, M=256, ws=A, wsb=need - 1) == Q.QUICK_ERR_WORKSPACE
    assert ex(cfg, M=256, ws=A + 4, wsb=need) == Q.QUICK_ERR_ALIGNMENT
    # stream-K: counters, then two fp32 partial tiles (128 x 256) per workgroup
    sk = Q.make_config(variant=3, tile_m=128, tile_n=32, split_k=64)
    assert Q.workspace_bytes(256, 4096, 4096, sk) == Q.WS_COUNTER_BYTES + 2 * 64 * 128 * 256 * 4
    # more workgroups than (tile, k-group) units: clamped to the units (2 x 16 x 32 = 1024)
    sk = Q.make_config(variant=3, tile_m=128, tile_n=32, split_k=4096)
    assert Q.workspace_bytes(256, 4096, 4096, sk) == Q.WS_COUNTER_BYTES + 2 * 1024 * 128 * 256 * 4
    # the reserved variant number: no plan, no workspace
    assert Q.workspace_bytes(1, 8192, 8192, Q.make_config(variant=4)) == 0
    # sliced stream kernel: counters, then 8 waves x n-tiles per wave x 1 KiB
    # per (column group, slice); slices raised to ceil(K/2048); one slice
    # needs none
    ks = Q.make_config(variant=5, split_k=8, tile_n=1)
    assert Q.workspace_bytes(16, 528, 8192, ks) == Q.WS_COUNTER_BYTES + 5 * 8 * 8 * 1024
    ks = Q.make_config(variant=5, split_k=1, tile_n=2)
    assert Q.workspace_bytes(16, 528, 8192, ks) == Q.WS_COUNTER_BYTES + 3 * 4 * 8 * 2 * 1024
    assert Q.workspace_bytes(16, 528, 2048, ks) == 0
    # automatic slices: the fewest (K / 2048 rounded up), two n-tiles per wave
    assert Q.workspace_bytes(1, 4096, 4096, Q.make_config(variant=5)) == Q.WS_COUNTER_BYTES + 16 * 2 * 8 * 2 * 1024
    # fewer than 8 units: one workgroup per tile, no workspace
    assert Q.workspace_bytes(16, 128, 512, Q.make_config(variant=3, tile_m=16, tile_n=16)) == 0


def test_grouped_validation_without_device():
    """Every argument check of the grouped entry point returns before any
    device work."""
    A = 0x10000
    L = Q.lib()

    def g(x=A, rows=A, offs=A, pw=A, ps=A, pz=A, y=A, T=64, R=128, E=8, N=4096, K=4096, group=128, cfg=None):
        if cfg is None:
            return L.quick_w4a16_grouped_gemm(x, rows, offs, pw, ps, pz, y, T, R, E, N, K, group, None)
        return L.quick_w4a16_grouped_gemm_ex(x, rows, offs, pw, ps, pz, y, T, R, E, N, K, group, None,
                                             ctypes.byref(cfg), None, 0)
    assert g(R=0) == Q.QUICK_OK
    assert g(0, 0, 0, 0, 0, 0, 0, R=0) == Q.QUICK_OK
    assert g(group=64) == Q.QUICK_ERR_UNSUPPORTED
    assert g(E=0) == Q.QUICK_ERR_SHAPE
    assert g(E=513) == Q.QUICK_ERR_SHAPE
    assert g(R=-1) == Q.QUICK_ERR_SHAPE
    assert g(T=-1) == Q.QUICK_ERR_SHAPE
    assert g(K=4000) == Q.QUICK_ERR_SHAPE
    assert g(N=4088) == Q.QUICK_ERR_SHAPE
    assert g(T=0) == Q.QUICK_ERR_SHAPE              # routed rows need token rows
    assert g(rows=0, T=64, R=128) == Q.QUICK_ERR_SHAPE   # identity rows need T >= R
    assert g(N=1 << 20, K=1 << 17) == Q.QUICK_ERR_SHAPE
    assert g(x=0) == Q.QUICK_ERR_INVALID_ARG
    assert g(offs=0) == Q.QUICK_ERR_INVALID_ARG
    assert g(y=0) == Q.QUICK_ERR_INVALID_ARG
    assert g(x=A + 8) == Q.QUICK_ERR_ALIGNMENT
    assert g(offs=A + 2) == Q.QUICK_ERR_ALIGNMENT
    assert g(rows=A + 2) == Q.QUICK_ERR_ALIGNMENT
    assert g(y=A + 4) == Q.QUICK_ERR_ALIGNMENT
    assert g(cfg=Q.make_config(variant=1)) == Q.QUICK_ERR_INVALID_ARG      # no stream kernel here
    assert g(cfg=Q.make_config(variant=4)) == Q.QUICK_ERR_INVALID_ARG
    assert g(cfg=Q.make_config(variant=2, tile_m=16, tile_n=64)) == Q.QUICK_ERR_INVALID_ARG
    assert g(cfg=Q.make_config(variant=2, split_k=33)) == Q.QUICK_ERR_INVALID_ARG
    assert g(cfg=Q.make_config(variant=3, split_k=12)) == Q.QUICK_ERR_INVALID_ARG
    # workspaces: split-K partials over all routed rows; stream-K slots per workgroup
    cfg = Q.make_config(variant=2, split_k=4, tile_m=64, tile_n=32)
    assert Q.grouped_workspace_bytes(1024, 8, 14336, 4096, cfg) == Q.WS_COUNTER_BYTES + 4 * 1024 * 14336 * 4
    cfg = Q.make_config(variant=3, split_k=64, tile_m=128, tile_n=32)
    assert Q.grouped_workspace_bytes(1024, 8, 14336, 4096, cfg) == Q.WS_COUNTER_BYTES + 2 * 64 * 128 * 256 * 4
    assert Q.grouped_workspace_bytes(1024, 8, 14336, 4096, Q.make_config(variant=2, tile_m=16, tile_n=16)) == 0
    assert Q.grouped_workspace_bytes(0, 8, 14336, 4096) == 0
    # the automatic full-height plan runs two stream-K launches (128-row tiles,
    # then 32-row tiles over short remainders): its workspace covers both, and
    # an all-zero cfg is the automatic choice
    main = Q.grouped_workspace_bytes(1024, 8, 14336, 4096, Q.make_config(variant=3, tile_m=128, tile_n=32))
    tail = Q.grouped_workspace_bytes(1024, 8, 14336, 4096, Q.make_config(variant=3, tile_m=32, tile_n=32))
    auto = Q.grouped_workspace_bytes(1024, 8, 14336, 4096)
    assert auto == max(main, tail) > 0
    assert Q.grouped_workspace_bytes(1024, 8, 14336, 4096, Q.make_config()) == auto


def test_fused_validation_without_device():
    """Argument checks of the fused entry points, and the plans the gated
    epilogue forces, before any device work."""
    A = 0x10000
    L = Q.lib()

    def f(act=1, bias=None, M=4, N=4096, K=4096, cfg=None):
        e = Q.QuickEpilogue(bias, act)
        return L.quick_w4a16_gemm_fused(A, A, A, A, A, M, N, K, 128, None, ctypes.byref(e),
                                        ctypes.byref(cfg) if cfg is not None else None, None, 0)
    assert f(M=0) == Q.QUICK_OK
    assert f(act=2) == Q.QUICK_ERR_INVALID_ARG
    assert f(N=4112) == Q.QUICK_ERR_SHAPE                     # gated: N a multiple of 32
    assert f(act=0, bias=A + 2) == Q.QUICK_ERR_ALIGNMENT
    # explicit configurations that cannot pair gate and up tiles in a wave
    assert f(cfg=Q.make_config(variant=1, split_k=4, tile_n=1)) == Q.QUICK_ERR_INVALID_ARG
    assert f(cfg=Q.make_config(variant=2, split_k=1, tile_m=16, tile_n=16)) == Q.QUICK_ERR_INVALID_ARG
    assert f(cfg=Q.make_config(variant=3, tile_m=32, tile_n=16)) == Q.QUICK_ERR_INVALID_ARG
    assert f(cfg=Q.make_config(variant=2, tile_m=64, tile_n=16)) == Q.QUICK_ERR_INVALID_ARG
    assert f(act=0, bias=A, cfg=Q.make_config(variant=4)) == Q.QUICK_ERR_INVALID_ARG
    # a split-K reduction applies the epilogue itself: 16-column waves are fine;
    # the gated output needs the same partials as the plain GEMM
    cfg = Q.make_config(variant=2, split_k=4, tile_m=16, tile_n=16)
    assert Q.fused_workspace_bytes(64, 4096, 4096, cfg, activation=1) == Q.workspace_bytes(64, 4096, 4096, cfg)
    # stream-K with the automatic 16-column tile moves to 32-column waves (bigger slots)
    sk = Q.make_config(variant=3, split_k=64, tile_m=16)
    assert Q.fused_workspace_bytes(64, 4096, 4096, sk, activation=1) == Q.WS_COUNTER_BYTES + 2 * 64 * 16 * 256 * 4
    # a per-expert bias cannot go through the split-K reduction
    e = Q.QuickEpilogue(A, 0)
    assert L.quick_w4a16_grouped_gemm_fused(A, A, A, A, A, A, A, 64, 128, 8, 4096, 4096, 128, None,
                                            ctypes.byref(e), ctypes.byref(Q.make_config(variant=2, split_k=2)),
                                            None, 0) == Q.QUICK_ERR_INVALID_ARG


def test_grouped_select_config():
    assert Q.grouped_select_config(1024, 8, 14336, 4096)["tile_m"] == 128   # ~128 rows per expert
    assert Q.grouped_select_config(64, 8, 14336, 4096)["tile_m"] == 16      # decode-sized batches
    c = Q.grouped_select_config(1024, 8, 4096, 14336)
    assert c["variant"] == Q.VARIANT_STREAMK and c["split_k"] % 8 == 0


def test_select_config_regimes():
    small = Q.select_config(1, 8192, 8192)
    large = Q.select_config(1024, 8192, 8192)
    assert small["variant"] == Q.VARIANT_STREAM
    assert large["variant"] == Q.VARIANT_TILED
    assert Q.workspace_bytes(1, 8192, 8192) == 0
    # 9 <= M <= 16: the sliced stream kernel (one n-tile per wave, the fewest
    # slices) unless it would have fewer than 128 workgroups or the weights
    # reach 128 MiB
    assert Q.select_config(16, 12288, 4096) == dict(variant=Q.VARIANT_KSTREAM, split_k=2, tile_m=0, tile_n=1)
    assert Q.select_config(9, 8192, 28672) == dict(variant=Q.VARIANT_KSTREAM, split_k=14, tile_m=0, tile_n=1)
    assert Q.select_config(16, 4096, 4096)["variant"] == Q.VARIANT_STREAM      # 32 x 2 workgroups
    assert Q.select_config(16, 57344, 8192)["variant"] == Q.VARIANT_TILED      # 224 MiB of weights
    # an explicit stream-kernel choice with its fields left 0 takes the stream defaults
    assert Q.workspace_bytes(16, 12288, 4096, Q.make_config(variant=1)) == 0


def test_status_strings():
    for st in range(9):
        assert Q.status_string(st).startswith("QUICK_")
    assert "unknown" in Q.status_string(99)


def test_tune_table_load_select_save(tmp_path):
    """A loaded tune table drives the automatic choice; save writes it back
    unchanged; a malformed file loads nothing."""
    Q.tune_table_clear()
    try:
        good = tmp_path / "t.txt"
        good.write_text("quick-tune 1\n256 4096 4096 2 4 64 32\n1 8192 8192 1 2 0 2\n"
                        "300 528 2304 3 24 64 32\n")
        Q.tune_table_load(str(good))
        assert Q.tune_table_size() == 3
        assert Q.select_config(256, 4096, 4096) == dict(variant=2, split_k=4, tile_m=64, tile_n=32)
        assert Q.select_config(1, 8192, 8192) == dict(variant=1, split_k=2, tile_m=0, tile_n=2)
        assert Q.select_config(300, 528, 2304)["variant"] == 3
        # the tuned split-K shape now needs its workspace in the automatic path too
        assert Q.workspace_bytes(256, 4096, 4096) == Q.WS_COUNTER_BYTES + 4 * 256 * 4096 * 4
        out = tmp_path / "u.txt"
        Q.tune_table_save(str(out))
        lines = out.read_text().splitlines()
        assert lines[0] == "quick-tune 1" and sorted(lines[1:]) == sorted(good.read_text().splitlines()[1:])
        for bad in ("quick-tune 2\n", "quick-tune 1\n256 4096 4096 2 4 64\n",
                    "quick-tune 1\n256 4096 4096 2 4 96 32\n", "quick-tune 1\n256 4096 4000 2 4 64 32\n",
                    "quick-tune 1\n1 2 3 4 5 6 7 8\n"):
            Q.tune_table_clear()
            f = tmp_path / "bad.txt"
            f.write_text(bad)
            with pytest.raises(Q.QuickError):
                Q.tune_table_load(str(f))
            assert Q.tune_table_size() == 0
        with pytest.raises(Q.QuickError):
            Q.tune_table_load(str(tmp_path / "missing.txt"))
    finally:
        Q.tune_table_clear()


def test_committed_tune_table_entries_are_valid_plans():
    """Every entry of the committed tune table is a configuration the
    planner accepts for its shape: with the table loaded, the automatic
    choice for each shape is that entry (an entry the planner rejected would
    fall back to the built-in rules)."""
    import os
    path = os.path.join(os.path.dirname(Q.__file__), "tune_mi355x.txt")
    lines = open(path).read().split("\n")
    assert lines[0] == "quick-tune 1"
    entries = [tuple(int(v) for v in l.split()) for l in lines[1:] if l.strip()]
    assert len(entries) == 44
    Q.tune_table_clear()
    try:
        Q.tune_table_load(path)
        assert Q.tune_table_size() == len(entries)
        for M, N, K, variant, split, tm, tn in entries:
            sel = Q.select_config(M, N, K)
            assert (sel["variant"], sel["tile_m"], sel["tile_n"]) == (variant, tm, tn), (M, N, K, sel)
            if variant == Q.VARIANT_STREAM:
                assert sel["split_k"] == split
    finally:
        Q.tune_table_clear()
