"""Library pack (host C++ in libquick.so) against the oracle's element-wise
definition of the QPK16 layout, byte for byte, plus round trip and errors."""
import numpy as np
import pytest

import oracle
import paper_2402_10076_amd as Q


def _weights(seed, K, N):
    g = np.random.Generator(np.random.PCG64(seed))
    q = g.integers(0, 16, (K, N), dtype=np.uint8)
    z = g.integers(0, 16, (K // 128, N), dtype=np.uint8)
    s = g.integers(0, 1 << 16, (K // 128, N), dtype=np.uint16)
    return q, z, s


SHAPES = [(128, 16), (256, 32), (384, 48), (1024, 80), (512, 272), (4096, 512)]


@pytest.mark.parametrize("K,N", SHAPES)
def test_pack_matches_oracle_definition(K, N):
    q, z, s = _weights(K * 7 + N, K, N)
    pw, ps, pz = Q.pack_weights(q, z, s)
    ow, oz, os_ = oracle.pack(q, z, s)
    assert pw.tobytes() == ow.tobytes()
    assert pz.tobytes() == oz.tobytes()
    assert ps.tobytes() == os_.tobytes()


@pytest.mark.parametrize("K,N", SHAPES)
def test_unpack_inverts_pack(K, N):
    q, z, s = _weights(K + N, K, N)
    pw, ps, pz = Q.pack_weights(q, z, s)
    q2, z2, s2 = Q.unpack_weights(pw, ps, pz, K, N)
    assert np.array_equal(q, q2) and np.array_equal(z, z2) and np.array_equal(s, s2)


def test_pack_sizes():
    assert Q.packed_sizes(4096, 4096) == (4096 * 4096 // 2, 4096 * 4096 // 256, 4096 * 4096 // 64)
    assert Q.pack_format_version() == 1


def test_index_encoded_permutation_matches_oracle():
    """Recover every nibble's source element through the library pack and
    require the same permutation as the oracle's definition."""
    K, N = 256, 48
    flat = np.arange(K * N, dtype=np.int64).reshape(K, N)
    z = np.zeros((K // 128, N), np.uint8)
    s = np.zeros((K // 128, N), np.uint16)
    lib_src = np.zeros(K * N, np.int64)
    orc_src = np.zeros(K * N, np.int64)
    for b in range(4):
        q = ((flat >> (4 * b)) & 15).astype(np.uint8)
        pw, _, _ = Q.pack_weights(q, z, s)
        ow, _, _ = oracle.pack(q, z, s)
        for src, words in ((lib_src, pw), (orc_src, ow)):
            nib = np.stack([(words >> (4 * i)) & 15 for i in range(8)], axis=1).reshape(-1)
            src |= nib.astype(np.int64) << (4 * b)
    assert np.array_equal(lib_src, orc_src)
    assert np.array_equal(np.sort(lib_src), np.arange(K * N))


def test_pack_errors_leave_outputs_untouched():
    K, N = 256, 32
    q, z, s = _weights(1, K, N)
    q[17, 5] = 16
    import ctypes
    wb, zb, sb = Q.packed_sizes(K, N)
    pw = np.full(wb // 4, 0xDEADBEEF, np.uint32)
    ps = np.full(sb // 2, 0xBEEF, np.uint16)
    pz = np.full(zb // 4, 0xDEADBEEF, np.uint32)
    P = lambda a: a.ctypes.data_as(ctypes.c_void_p)
    rc = Q.lib().quick_pack_weights(P(q), P(z), P(s), K, N, 128, P(pw), P(ps), P(pz))
    assert rc == Q.QUICK_ERR_RANGE
    assert np.all(pw == 0xDEADBEEF) and np.all(ps == 0xBEEF) and np.all(pz == 0xDEADBEEF)
    q[17, 5] = 3
    z[1, 2] = 200
    assert Q.lib().quick_pack_weights(P(q), P(z), P(s), K, N, 128, P(pw), P(ps), P(pz)) == Q.QUICK_ERR_RANGE
    z[1, 2] = 0
    assert Q.lib().quick_pack_weights(P(q), P(z), P(s), K, N, 64, P(pw), P(ps), P(pz)) == Q.QUICK_ERR_UNSUPPORTED
    assert Q.lib().quick_pack_weights(P(q), P(z), P(s), 200, N, 128, P(pw), P(ps), P(pz)) == Q.QUICK_ERR_SHAPE
    assert Q.lib().quick_pack_weights(P(q), P(z), P(s), K, 24, 128, P(pw), P(ps), P(pz)) == Q.QUICK_ERR_SHAPE
    assert Q.lib().quick_pack_weights(None, P(z), P(s), K, N, 128, P(pw), P(ps), P(pz)) == Q.QUICK_ERR_INVALID_ARG
    with pytest.raises(Q.QuickError):
        Q.pack_weights(np.full((K, N), 16, np.uint8), z, s)


def test_interleave_gate_up_matches_oracle_layout():
    """The library's gate/up column interleave equals the oracle's, byte for
    byte, for q, z and s."""
    g = np.random.Generator(np.random.PCG64(31))
    K, Nh = 256, 48
    gate = (g.integers(0, 16, (K, Nh), dtype=np.uint8), g.integers(0, 16, (K // 128, Nh), dtype=np.uint8),
            g.integers(0, 1 << 15, (K // 128, Nh)).astype(np.uint16))
    up = (g.integers(0, 16, (K, Nh), dtype=np.uint8), g.integers(0, 16, (K // 128, Nh), dtype=np.uint8),
          g.integers(0, 1 << 15, (K // 128, Nh)).astype(np.uint16))
    q, z, s = Q.interleave_gate_up(gate, up)
    for got, a, b in zip((q, z, s), gate, up):
        assert np.array_equal(got, oracle.interleave_gate_up(a, b))


def test_tile_decode_inverts_oracle_pack():
    """The tests' decoder of one n-tile's QPK16 words (used where inputs are
    drawn on the device in packed form) against the oracle's definition."""
    from gpu_util import decode_qpk16_tile
    K, N = 512, 64
    q, z, s = _weights(99, K, N)
    ow, oz, os_ = oracle.pack(q, z, s)
    KG = K // 128
    for nt in range(N // 16):
        dq, dz, ds = decode_qpk16_tile(ow[nt * KG * 256:(nt + 1) * KG * 256], oz[nt * KG * 2:(nt + 1) * KG * 2],
                                       os_[nt * KG * 16:(nt + 1) * KG * 16], K)
        cols = slice(16 * nt, 16 * nt + 16)
        assert np.array_equal(dq, q[:, cols]) and np.array_equal(dz, z[:, cols]) and np.array_equal(ds, s[:, cols])
