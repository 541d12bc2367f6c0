"""The largest shapes the kernels' 32-bit offsets admit (the host rejects
anything larger: packed weights of 4 GiB or more, activations or outputs of
2^31 elements or more), each run on several plans and checked against the
oracle on sampled tiles or rows:

* weights just under 4 GiB (K = 65536, N = 131056): every unit offset of the
  last n-tiles sits just below 2^32 bytes;
* activations just under 2^31 elements (M = 524287 rows of K = 4096);
* outputs just under 2^31 elements (M = 65535 rows of N = 32752);
* the grouped form over 8 experts of 1 GiB each, whose buffers start beyond
  2^32 bytes.

Inputs of this size are drawn on the device with a seeded torch generator:
x as normal f16, the packed weights and zero points as uniform random bytes
(every byte holds two valid 4-bit codes), the scales as f16 in [0.002, 0.02).
The oracle gets what the samples need, copied to the host: rows of x, and the
weights of the sampled n-tiles decoded from their QPK16 words; each decoded
tile is re-packed by the oracle's pack and must reproduce those words byte
for byte, so the oracle's inputs follow the layout's definition."""
import numpy as np
import pytest
import torch

import oracle
import paper_2402_10076_amd as Q
from gpu_util import TOL, decode_qpk16_tile, from_dev_y, rand_case, rel_err, say

pytestmark = pytest.mark.gpu


def _gen(seed):
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    return g


def _dev_weights(seed, K, N, experts=1):
    """Random packed weights, zero points and scales of `experts` K x N
    matrices back to back, on the device."""
    g = _gen(seed)
    wb, zb, sb = (experts * b for b in Q.packed_sizes(K, N))   # packed, zero-point and scale bytes
    pw = torch.randint(0, 256, (wb,), dtype=torch.uint8, device="cuda", generator=g).view(torch.int32)
    pz = torch.randint(0, 256, (zb,), dtype=torch.uint8, device="cuda", generator=g).view(torch.int32)
    ps = (torch.rand(sb // 2, device="cuda", generator=g) * 0.018 + 0.002).half().view(torch.int16)
    return pw, ps, pz


def _host_tile(pw, ps, pz, K, nt):
    """(q, z, s) of n-tile nt, decoded from the device words and checked
    against the oracle's pack of the decoded values."""
    KG = K // 128
    w = pw[nt * KG * 256:(nt + 1) * KG * 256].cpu().numpy().view(np.uint32)
    z = pz[nt * KG * 2:(nt + 1) * KG * 2].cpu().numpy().view(np.uint32)
    s = ps[nt * KG * 16:(nt + 1) * KG * 16].cpu().numpy().view(np.uint16)
    q_t, z_t, s_t = decode_qpk16_tile(w, z, s, K)
    ow, oz, os_ = oracle.pack(q_t, z_t, s_t)
    assert ow.tobytes() == w.tobytes() and oz.tobytes() == z.tobytes() and os_.tobytes() == s.tobytes()
    return q_t, z_t, s_t


def _cfg(c):
    return Q.make_config(**c) if c else None


def _cid(c):
    if c is None:
        return "auto"
    return "v%d_s%d_%dx%d" % (c["variant"], c["split_k"], c.get("tile_m", 0), c["tile_n"])


BIG_W = [None, dict(variant=1, split_k=8, tile_n=2), dict(variant=5, split_k=0, tile_n=1),
         dict(variant=2, split_k=1, tile_m=16, tile_n=16), dict(variant=2, split_k=4, tile_m=16, tile_n=32),
         dict(variant=3, split_k=0, tile_m=16, tile_n=16)]


def test_largest_weights():
    """K x N / 2 = 4,294,443,008 bytes of packed weights, M = 5."""
    M, K, N = 5, 65536, 131056
    assert K * N // 2 < 1 << 32 <= K * (N + 16) // 2   # the next N is rejected
    say("largest weights: M=%d K=%d N=%d" % (M, K, N))
    pw, ps, pz = _dev_weights(11, K, N)
    x = torch.randn(M, K, device="cuda", generator=_gen(12), dtype=torch.float16)
    xb = x.cpu().view(torch.int16).numpy().view(np.uint16)
    NT, KG = N // 16, K // 128
    # first tiles, the tile holding byte 2^31 of the packed weights, the last tiles, and random ones
    tiles = sorted(set([0, 1, (1 << 31) // (KG * 1024), NT - 2, NT - 1] +
                       list(np.random.Generator(np.random.PCG64(13)).integers(0, NT, 3))))
    refs = {}
    for nt in tiles:
        q_t, z_t, s_t = _host_tile(pw, ps, pz, K, nt)
        refs[nt] = oracle.gemm(xb, q_t, z_t, s_t)
    for c in BIG_W:
        say("  plan %s" % _cid(c))
        y = from_dev_y(Q.w4a16_gemm(x, pw, ps, pz, N, cfg=_cfg(c)))
        for nt in tiles:
            err = rel_err(y[:, 16 * nt:16 * nt + 16], refs[nt])
            assert err <= TOL, "plan %s, n-tile %d: %.3g" % (_cid(c), nt, err)
    del pw, ps, pz
    torch.cuda.empty_cache()


BIG_X = [None, dict(variant=2, split_k=1, tile_m=128, tile_n=32), dict(variant=6, split_k=1, tile_m=128, tile_n=32),
         dict(variant=3, split_k=0, tile_m=128, tile_n=16), dict(variant=2, split_k=2, tile_m=64, tile_n=16),
         dict(variant=7, split_k=0, tile_m=64, tile_n=32)]


def _sample_rows(M, marks, seed, n):
    r = set(int(v) for v in marks if 0 <= v < M)
    r.update(int(v) for v in np.random.Generator(np.random.PCG64(seed)).integers(0, M, n))
    return np.array(sorted(r), np.int64)


def test_largest_activations():
    """M x K = 2^31 - 4096 activation elements (4 GiB of x), N = 48."""
    K, N = 4096, 48
    M = (1 << 31) // K - 1
    say("largest activations: M=%d K=%d N=%d" % (M, K, N))
    _, q, z, s = rand_case(21, 16, K, N)
    pw, ps, pz = Q.to_device(*Q.pack_weights(q, z, s))
    x = torch.randn(M, K, device="cuda", generator=_gen(22), dtype=torch.float16)
    half = (1 << 30) // K   # rows whose byte offsets cross 2^31
    rows = _sample_rows(M, [0, 1, half - 1, half, half + 1, M - 2, M - 1], 23, 57)
    ref = oracle.gemm(x[torch.from_numpy(rows).cuda()].cpu().view(torch.int16).numpy().view(np.uint16), q, z, s)
    for c in BIG_X:
        say("  plan %s" % _cid(c))
        y = Q.w4a16_gemm(x, pw, ps, pz, N, cfg=_cfg(c))
        yr = from_dev_y(y[torch.from_numpy(rows).cuda()])
        err = rel_err(yr, ref)
        assert err <= TOL, "plan %s: %.3g" % (_cid(c), err)
        del y
    del x
    torch.cuda.empty_cache()


BIG_Y = [None, dict(variant=2, split_k=1, tile_m=64, tile_n=32), dict(variant=6, split_k=1, tile_m=128, tile_n=32),
         dict(variant=2, split_k=1, tile_m=16, tile_n=16), dict(variant=3, split_k=0, tile_m=128, tile_n=32)]


def test_largest_outputs():
    """M x N = 2,146,402,320 output elements (4 GiB of y), K = 128."""
    M, K, N = 65535, 128, 32752
    assert M * N < 1 << 31
    say("largest outputs: M=%d K=%d N=%d" % (M, K, N))
    _, q, z, s = rand_case(31, 16, K, N)
    pw, ps, pz = Q.to_device(*Q.pack_weights(q, z, s))
    x = torch.randn(M, K, device="cuda", generator=_gen(32), dtype=torch.float16)
    mid = (1 << 30) // N    # rows whose output offsets cross 2^31 bytes
    rows = _sample_rows(M, [0, 1, mid - 1, mid, mid + 1, M - 2, M - 1], 33, 17)
    ref = oracle.gemm(x[torch.from_numpy(rows).cuda()].cpu().view(torch.int16).numpy().view(np.uint16), q, z, s)
    for c in BIG_Y:
        say("  plan %s" % _cid(c))
        y = Q.w4a16_gemm(x, pw, ps, pz, N, cfg=_cfg(c))
        yr = from_dev_y(y[torch.from_numpy(rows).cuda()])
        err = rel_err(yr, ref)
        assert err <= TOL, "plan %s: %.3g" % (_cid(c), err)
        del y
    del x
    torch.cuda.empty_cache()


BIG_E = [None, dict(variant=2, split_k=1, tile_m=16, tile_n=16), dict(variant=2, split_k=1, tile_m=32, tile_n=32),
         dict(variant=3, split_k=16, tile_m=64, tile_n=32), dict(variant=2, split_k=3, tile_m=16, tile_n=16)]


def test_grouped_experts_beyond_4gib():
    """Grouped form over 8 experts of 1 GiB of packed weights each (8 GiB
    back to back, so the later experts' buffers start beyond 2^32 bytes),
    gathered token rows, empty experts included."""
    K, N, E, T = 32768, 65536, 8, 64
    counts = [3, 0, 5, 1, 7, 2, 0, 9]
    say("grouped, 8 x 1 GiB experts: K=%d N=%d" % (K, N))
    pw, ps, pz = _dev_weights(41, K, N, experts=E)
    x = torch.randn(T, K, device="cuda", generator=_gen(42), dtype=torch.float16)
    xb = x.cpu().view(torch.int16).numpy().view(np.uint16)
    g = np.random.Generator(np.random.PCG64(43))
    rows = g.integers(0, T, sum(counts)).astype(np.int32)
    offsets = np.concatenate([[0], np.cumsum(counts)]).astype(np.int32)
    NT, KG = N // 16, K // 128
    wb, zb, sb = Q.packed_sizes(K, N)
    tiles = [0, NT - 1, int(g.integers(1, NT - 1))]
    refs = {}
    for e in range(E):
        lo, hi = int(offsets[e]), int(offsets[e + 1])
        if hi == lo:
            continue
        # expert e's buffers start wb, sb, zb bytes after expert e-1's
        we, se, ze = pw[e * wb // 4:(e + 1) * wb // 4], ps[e * sb // 2:(e + 1) * sb // 2], pz[e * zb // 4:(e + 1) * zb // 4]
        for nt in tiles:
            q_t, z_t, s_t = _host_tile(we, se, ze, K, nt)
            refs[(e, nt)] = oracle.gemm(xb[rows[lo:hi]], q_t, z_t, s_t)
    od, rd = torch.from_numpy(offsets).cuda(), torch.from_numpy(rows).cuda()
    for c in BIG_E:
        say("  plan %s" % _cid(c))
        y = from_dev_y(Q.grouped_gemm(x, od, pw, ps, pz, N, rows=rd, cfg=_cfg(c)))
        for (e, nt), ref in refs.items():
            lo, hi = int(offsets[e]), int(offsets[e + 1])
            err = rel_err(y[lo:hi, 16 * nt:16 * nt + 16], ref)
            assert err <= TOL, "plan %s, expert %d, n-tile %d: %.3g" % (_cid(c), e, nt, err)
    del pw, ps, pz
    torch.cuda.empty_cache()
