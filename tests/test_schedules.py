"""Host-side checks of the GEMM schedules, without a GPU.

* The library's own planning through the C ABI: for many shapes the
  automatic configuration is one the explicit path accepts, and the
  workspace the automatic path reports equals the one of that explicit
  configuration.
* The index arithmetic of the persistent schedules, written out the way the
  kernels compute it: the stream-K schedule (whole rounds of tiles, then the
  rest of tiles x k-groups split), the grouped form's per-expert tile table,
  and the sliced stream kernel's slices.  Each must cover every unit exactly
  once, give every shared tile a
  contiguous run of contributors whose partial-slot indices agree between
  writer and reader, and keep every access inside its buffer.  (These are the
  checks run before each schedule first ran on a GPU.)
"""
import numpy as np
import pytest

import paper_2402_10076_amd as Q


@pytest.mark.parametrize("seed", range(4))
def test_automatic_plans_are_valid_explicit_plans(seed):
    g = np.random.Generator(np.random.PCG64(seed))
    for _ in range(60):
        M = int(g.choice([1, 2, 4, 8, 9, 16, 17, 33, 64, 65, 100, 128, 200, 256, 512, 1024, 2048]))
        N = int(g.integers(1, 512)) * 16
        K = int(g.integers(1, 128)) * 128
        sel = Q.select_config(M, N, K)
        cfg = Q.make_config(**sel)
        assert Q.workspace_bytes(M, N, K, cfg) == Q.workspace_bytes(M, N, K), (M, N, K, sel)
        assert sel["variant"] in (Q.VARIANT_STREAM, Q.VARIANT_TILED, Q.VARIANT_STREAMK, Q.VARIANT_KSTREAM), sel
        if sel["variant"] == Q.VARIANT_KSTREAM:
            assert 9 <= M <= 16 and sel["split_k"] == -(-K // 2048)


def _owner(u, W, U):
    """Worker owning unit u when W workers split U units as [w*U/W, (w+1)*U/W)."""
    return ((u + 1) * W - 1) // U


def streamk_dp_tiles(tiles, KG, G):
    """Tiles the stream-K schedule runs whole, one per workgroup, before it
    splits the rest: the whole rounds, less one when the remainder would
    give each workgroup under half a tile (or under one k-group)."""
    tdp = tiles // G * G
    if 0 < tdp < tiles and (2 * (tiles - tdp) < G or (tiles - tdp) * KG < G):
        tdp -= G
    return tdp


def streamk_partition(tiles, KG, G):
    """Stream-K of the tiled kernel: G workgroups (8 <= G <= tiles*KG, a
    multiple of 8) first run tiles wid, wid + G, .. below streamk_dp_tiles
    whole, then split the remaining tiles x KG units; returns per tile the
    contributor list [(workgroup, slot, kb, ke)] in k order, and the first
    unit and the unit count of the split part."""
    tdp = streamk_dp_tiles(tiles, KG, G)
    pieces = {}
    for wid in range(G):
        for t in range(wid, tdp, G):
            pieces.setdefault(t, []).append((wid, None, 0, KG))
    ub = tdp * KG
    U = tiles * KG - ub
    for wid in range(G if U else 0):   # whole rounds only: nothing is split
        u0, u1 = ub + wid * U // G, ub + (wid + 1) * U // G
        assert u1 > u0, "empty range"
        u = u0
        while u < u1:
            tt, kb = divmod(u, KG)
            ke = min(KG, kb + (u1 - u))
            if not (kb == 0 and ke == KG):
                slot = 2 * wid + (0 if u == u0 else 1)
                assert slot < 2 * G
                pieces.setdefault(tt, []).append((wid, slot, kb, ke))
            else:
                pieces.setdefault(tt, []).append((wid, None, 0, KG))
            u += ke - kb
    return pieces, ub, U


@pytest.mark.parametrize("tiles,KG,G", [(1, 32, 8), (3, 7, 16), (40, 64, 256), (256, 224, 256), (320, 64, 256),
                                         (17, 9, 152), (5, 200, 1000), (896, 64, 256), (36, 8, 16), (40, 8, 16),
                                         (60, 8, 16), (16, 8, 16), (25, 3, 24), (1792, 64, 256), (300, 1, 256)])
def test_streamk_contributors_and_slots(tiles, KG, G):
    G = min(G, tiles * KG) // 8 * 8
    pieces, ub, U = streamk_partition(tiles, KG, G)
    assert sorted(pieces) == list(range(tiles))
    tdp = streamk_dp_tiles(tiles, KG, G)
    assert tdp % G == 0 and 0 <= tdp <= tiles
    if tdp < tiles:
        # the split part gives every workgroup at least one k-group and,
        # after whole rounds, between half a tile and 3/2 tiles
        assert U >= G
        if tdp:
            assert G <= 2 * (tiles - tdp) < 3 * G
    for t, ps in pieces.items():
        # the k-ranges of a tile's pieces tile [0, KG) in contributor order
        assert [p[2] for p in ps][0] == 0 and ps[-1][3] == KG
        assert all(a[3] == b[2] for a, b in zip(ps, ps[1:]))
        if t < tdp:
            assert ps == [(t % G, None, 0, KG)]
        if len(ps) == 1:
            continue
        tb = t * KG - ub
        w0, w1 = _owner(tb, G, U), _owner(tb + KG - 1, G, U)
        assert [p[0] for p in ps] == list(range(w0, w1 + 1)), "contributors are consecutive"
        for wid, slot, _, _ in ps:
            # the reader's rule for a contributor's slot
            assert slot == 2 * wid + (0 if wid * U // G >= tb else 1)
    # one arrival counter per workgroup: the owner of a split tile's last
    # unit owns no other split tile's last unit
    lasts = [_owner(t * KG - ub + KG - 1, G, U) for t, ps in pieces.items() if len(ps) > 1]
    assert len(lasts) == len(set(lasts)) and all(0 <= w < G for w in lasts)


def grouped_tiles(offsets, R, BM, nn, part=0, unit=128, keep=64):
    """The grouped kernel's tile table (clamped offsets, the rows of this
    launch's part, per-expert m-tile counts, prefix sums) and its tile ->
    (expert, m0, mend, n-tile) map."""
    E = len(offsets) - 1
    lo, hi, cum = [], [], [0]
    for e in range(E):
        a = min(max(offsets[e], 0), R)
        b = min(max(offsets[e + 1], a), R)
        if part:
            rem = (b - a) % unit
            lead = b if rem >= keep else b - rem
            if part == 1:
                b = lead
            else:
                a = lead
        lo.append(a), hi.append(b), cum.append(cum[-1] + (b - a + BM - 1) // BM)

    def tile(t):
        a, b = 0, E
        while b - a > 1:
            mid = (a + b) // 2
            if cum[mid] * nn <= t:
                a = mid
            else:
                b = mid
        e = a
        local = t - cum[e] * nn
        te = cum[e + 1] - cum[e]
        nt = local // te
        m0 = lo[e] + (local - nt * te) * BM
        return e, m0, hi[e], nt
    return cum[E], tile


@pytest.mark.parametrize("counts,BM", [([130, 149, 111, 127, 132, 133, 122, 120], 128), ([0, 0, 5, 0], 16),
                                        ([37, 0, 129, 1, 66], 64), ([1], 32), ([3] * 300, 16)])
def test_grouped_tile_table_covers_every_row_once(counts, BM):
    offsets = np.concatenate([[0], np.cumsum(counts)]).tolist()
    R = offsets[-1]
    nn = 3
    n_mt, tile = grouped_tiles(offsets, R, BM, nn)
    assert n_mt <= (R + len(counts) * (BM - 1)) // BM, "host upper bound of m-tiles"
    seen = np.zeros((R, nn), np.int64)
    for t in range(n_mt * nn):
        e, m0, mend, nt = tile(t)
        assert offsets[e] <= m0 < mend <= offsets[e + 1] and nt < nn
        seen[m0:min(m0 + BM, mend), nt] += 1
    assert np.all(seen == 1)


@pytest.mark.parametrize("counts", [[130, 149, 111, 127, 132, 133, 122, 120], [20, 0, 257, 128, 200, 63, 64, 1],
                                    [0, 0, 0], [300], [127, 129, 191, 192, 193]])
def test_grouped_two_part_split_covers_every_row_once(counts):
    """The automatic full-height grouped plan runs as two launches: 128-row
    tiles over each expert's whole tiles (and a remainder of >= 64 rows),
    then 32-row tiles over the short remainders.  Together they cover every
    routed row once; the second part holds fewer than 64 rows per expert."""
    offsets = np.concatenate([[0], np.cumsum(counts)]).tolist()
    R = offsets[-1]
    nn = 2
    seen = np.zeros((max(R, 1), nn), np.int64)
    for part, BM in ((1, 128), (2, 32)):
        n_mt, tile = grouped_tiles(offsets, R, BM, nn, part=part)
        per_expert = {}
        for t in range(n_mt * nn):
            e, m0, mend, nt = tile(t)
            assert offsets[e] <= m0 < mend <= offsets[e + 1]
            rows = min(m0 + BM, mend) - m0
            seen[m0:m0 + rows, nt] += 1
            per_expert[e] = per_expert.get(e, 0) + rows
        if part == 2:
            assert all(v < 2 * 64 for v in per_expert.values())     # nn n-tiles x < 64 rows
    assert np.all(seen[:R] == 1)


def test_grouped_tile_table_clamps_malformed_offsets():
    """Decreasing or out-of-range offsets stay inside [0, R)."""
    R, BM, nn = 50, 16, 2
    for offsets in ([0, 70, 20, 50], [-5, 10, 10, 99], [0, 50, 40, 30]):
        n_mt, tile = grouped_tiles(offsets, R, BM, nn)
        for t in range(n_mt * nn):
            e, m0, mend, nt = tile(t)
            assert 0 <= m0 < mend <= R


def kstream_partition(M, N, K, npw, split):
    """Sliced stream kernel: the host's slice count and grid, then, per
    workgroup id, the kernel's (slice, column group), its waves' n-tiles and
    k-groups, its slice copy and its partial slots."""
    KG, NT = K // 128, N // 16
    kmax = 16
    smin = -(-KG // kmax)
    S = min(max(split, smin), KG)
    kgps = -(-KG // S)
    S = -(-KG // kgps)
    ncg = -(-NT // (8 * npw))
    G = ncg * S
    grid = -(-G // 8) * 8
    lds = -(-(M * kgps) // 4) * 1024
    assert lds <= 64 * 1024
    wg_bytes = 8 * npw * 1024
    covered = np.zeros((NT, KG), np.int64)
    slots = set()
    for b in range(grid):
        t = (b & 7) * (grid >> 3) + (b >> 3)
        if t >= G:
            continue
        s, cg = divmod(t, ncg)
        kb = s * kgps
        nk = min(KG, kb + kgps) - kb
        assert 1 <= nk <= kmax
        chunks = M * nk * 16
        for wave in range(8):
            i0 = wave * 64
            while i0 < chunks:
                for lane in range(64):
                    idx = min(i0 + lane, chunks - 1)
                    row, q = divmod(idx, nk * 16)
                    qs = (q & ~15) | ((q ^ row) & 15)
                    assert 0 <= (row * K + kb * 128 + qs * 8) * 2 < M * K * 2   # source inside x
                    assert (i0 + lane) * 16 + 16 <= lds                         # destination inside the LDS
                i0 += 64 * 8
            for p in range(npw):
                nt = cg * 8 * npw + wave * npw + p
                if nt < NT:
                    covered[nt, kb:kb + nk] += 1
                if S > 1:
                    off = (cg * S + s) * wg_bytes + (wave * npw + p) * 1024
                    assert off + 1024 <= G * wg_bytes and off not in slots
                    slots.add(off)
    assert (covered == 1).all()
    assert ncg <= 4096 and G * wg_bytes < 2 ** 32
    return S, kgps


@pytest.mark.parametrize("M,N,K,npw,split", [(16, 272, 4096, 1, 0), (16, 272, 4096, 2, 7), (3, 80, 2304, 1, 7),
                                             (9, 528, 6144, 2, 1), (1, 16, 128, 1, 0), (16, 48, 28672, 2, 0),
                                             (16, 4096, 11008, 1, 12), (16, 12288, 4096, 1, 0)])
def test_kstream_slices_cover_every_unit_once(M, N, K, npw, split):
    S, kgps = kstream_partition(M, N, K, npw, split)
    cfg = Q.make_config(variant=Q.VARIANT_KSTREAM, split_k=split, tile_n=npw)
    want = 0 if S == 1 else Q.WS_COUNTER_BYTES + -(-(N // 16) // (8 * npw)) * S * 8 * npw * 1024
    assert Q.workspace_bytes(M, N, K, cfg) == want
