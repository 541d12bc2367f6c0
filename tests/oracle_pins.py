"""Pins for the CPU oracle: checks against facts that do not come from the
oracle itself.

Each ``pin_*`` function raises AssertionError when the oracle disagrees with
what the mathematics or an independent routine fixes:

* binary16 decode/encode against numpy's float16 conversions (an IEEE 754
  library implementation), over all 65536 patterns and over rounding ties;
* the integer special case s = 1, z = 0, integer x: the GEMM must equal an
  int64 matrix product exactly;
* the closed form for weights that are constant down each column inside a
  group, y[m][n] = sum_g (c_n - z[g][n]) s[g][n] R[m][g] with R the group sums
  of x (exercises the group index, the zero point and the scale);
* an exact rational brute force (fractions.Fraction) on tiny shapes, with
  the oracle inside the worst-case binary64 summation bound;
* z == q  =>  y == 0 exactly; doubling every scale doubles y exactly;
* dequant() equals the GEMM of an identity activation matrix;
* the packed layout: hand-derived (word, nibble) positions of single
  elements, and that the layout is a bijection of the K*N nibbles.

The same functions are run against deliberately broken builds of oracle.c in
test_oracle.py, so every planted mistake must trip at least one of them.
"""
from __future__ import annotations

from fractions import Fraction

import numpy as np

import oracle

ONE_F16 = 0x3C00


def _rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def _f16(a):
    return np.asarray(a, np.float64).astype(np.float16).view(np.uint16)


def _rand_case(seed, M, K, N, group=128):
    g = _rng(seed)
    x = _f16(g.standard_normal((M, K)))
    q = g.integers(0, 16, (K, N), dtype=np.uint8)
    z = g.integers(0, 16, (K // group, N), dtype=np.uint8)
    s = _f16(g.uniform(0.002, 0.02, (K // group, N)))
    return x, q, z, s


# ---------------------------------------------------------------- binary16

def pin_f16_decode_all():
    bits = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    got = oracle.f16_to_f64(bits)
    ref = bits.view(np.float16).astype(np.float64)
    nan = np.isnan(ref)
    assert np.array_equal(np.isnan(got), nan), "NaN patterns differ"
    assert np.array_equal(got[~nan], ref[~nan]), "binary16 decode differs from IEEE 754"
    # signed zero
    assert np.array_equal(np.signbit(got[~nan]), np.signbit(ref[~nan]))


def pin_f16_encode():
    g = _rng(11)
    vals = [g.standard_normal(20000) * 10.0 ** g.integers(-9, 6, 20000),
            g.uniform(-70000, 70000, 5000)]
    # exact ties halfway between neighbouring binary16 values, incl. subnormals
    b = np.arange(0, 0x7bff, 7, dtype=np.uint16)
    lo = b.view(np.float16).astype(np.float64)
    hi = (b + 1).view(np.float16).astype(np.float64)
    vals.append((lo + hi) / 2)
    vals.append(-(lo + hi) / 2)
    vals.append(np.array([0.0, -0.0, 2.0 ** -25, 2.0 ** -25 * (1 + 2 ** -40), 2.0 ** -24,
                          1.5 * 2.0 ** -24, 2.0 ** -14, 65504.0, 65519.99, 65520.0, 1e6,
                          np.inf, -np.inf, 1.0 + 2.0 ** -11, 1.0 + 3 * 2.0 ** -11]))
    v = np.concatenate(vals)
    got = oracle.f64_to_f16(v)
    with np.errstate(over="ignore"):
        ref = v.astype(np.float16).view(np.uint16)
    assert np.array_equal(got, ref), "binary16 rounding differs at %d values" % int((got != ref).sum())
    assert oracle.f64_to_f16(np.array([np.nan]))[0] & 0x7c00 == 0x7c00


# ---------------------------------------------------------------- GEMM

def pin_integer_case():
    """s = 1, z = 0 and integer-valued x: every product and partial sum is an
    integer far below 2^53, so the binary64 GEMM must equal int64 exactly."""
    for seed, (M, K, N) in enumerate([(5, 256, 48), (1, 384, 16), (3, 128, 32)]):
        g = _rng(100 + seed)
        xi = g.integers(-4, 5, (M, K))
        q = g.integers(0, 16, (K, N), dtype=np.uint8)
        z = np.zeros((K // 128, N), np.uint8)
        s = np.full((K // 128, N), ONE_F16, np.uint16)
        y = oracle.gemm(_f16(xi), q, z, s)
        ref = xi.astype(np.int64) @ q.astype(np.int64)
        assert np.array_equal(y, ref.astype(np.float64)), "integer GEMM mismatch"


def pin_closed_form():
    """q constant down each column: y[m][n] = sum_g (c_n - z[g][n]) s[g][n] R[m][g]."""
    for seed, (M, K, N) in enumerate([(4, 512, 48), (2, 256, 16)]):
        g = _rng(200 + seed)
        G = K // 128
        x = _f16(g.standard_normal((M, K)))
        c = g.integers(0, 16, N)
        q = np.broadcast_to(c.astype(np.uint8), (K, N)).copy()
        z = g.integers(0, 16, (G, N), dtype=np.uint8)
        s = _f16(g.uniform(0.002, 0.02, (G, N)))
        xf = x.view(np.float16).astype(np.float64)
        sf = s.view(np.float16).astype(np.float64)
        R = xf.reshape(M, G, 128).sum(axis=2)              # [M][G]
        coef = (c[None, :] - z.astype(np.int64)) * sf       # [G][N]
        ref = R @ coef
        y = oracle.gemm(x, q, z, s)
        scale = np.abs(R) @ np.abs(coef) + 1e-300
        assert np.all(np.abs(y - ref) <= 1e-12 * scale), "closed form mismatch"


def pin_exact_fraction():
    """Exact rational evaluation of the definition on tiny shapes; the binary64
    oracle must lie within K * 2^-52 * sum|terms| of it."""
    for seed, (M, K, N) in enumerate([(3, 128, 16), (2, 256, 32), (1, 128, 32)]):
        x, q, z, s = _rand_case(300 + seed, M, K, N)
        xf = [[Fraction(float(v)) for v in row] for row in x.view(np.float16)]
        sf = [[Fraction(float(v)) for v in row] for row in s.view(np.float16)]
        y = oracle.gemm(x, q, z, s)
        for m in range(M):
            for n in range(N):
                tot = Fraction(0)
                mag = Fraction(0)
                for k in range(K):
                    t = xf[m][k] * (int(q[k, n]) - int(z[k // 128, n])) * sf[k // 128][n]
                    tot += t
                    mag += abs(t)
                bound = float(mag) * K * 2.0 ** -52
                assert abs(y[m, n] - float(tot)) <= bound, "exact brute force mismatch at (%d,%d)" % (m, n)


def pin_grouped_exact_fraction():
    """The mixture-of-experts form on a tiny case, by exact rational
    arithmetic written out per routed row: 3 experts (one owning no rows),
    gathered token rows with repeats and out of order."""
    g = _rng(410)
    T, K, N = 5, 128, 16
    x = _f16(g.standard_normal((T, K)))
    experts = []
    for e in range(3):
        experts.append((g.integers(0, 16, (K, N), dtype=np.uint8), g.integers(0, 16, (1, N), dtype=np.uint8),
                        _f16(g.uniform(0.002, 0.02, (1, N)))))
    offsets = [0, 3, 3, 7]               # expert 1 owns no rows
    rows = [4, 0, 4, 2, 1, 3, 0]
    y = oracle.grouped_gemm(x, rows, offsets, experts)
    assert y.shape == (7, N)
    xf = [[Fraction(float(v)) for v in r] for r in x.view(np.float16)]
    for r in range(7):
        e = 0 if r < 3 else 2
        q, z, s = experts[e]
        for n in range(N):
            sf = Fraction(float(s.view(np.float16)[0, n]))
            tot = Fraction(0)
            mag = Fraction(0)
            for k in range(K):
                t = xf[rows[r]][k] * (int(q[k, n]) - int(z[0, n])) * sf
                tot += t
                mag += abs(t)
            assert abs(y[r, n] - float(tot)) <= float(mag) * K * 2.0 ** -52, "grouped mismatch at (%d,%d)" % (r, n)


def pin_epilogue_invariants():
    """The fused epilogue against facts of the mathematics: silu(a) - silu(-a)
    = a (a*sigmoid(a) + a*sigmoid(-a) = a), silu(0) = 0, silu(a) -> a for
    large a and -> 0 for very negative a; an up factor of 1 leaves silu
    alone; a bias adds exactly its binary16 value; and the tile layout maps
    gate column 32t+i and up column 32t+16+i to output 16t+i."""
    g = _rng(420)
    M, Nh = 3, 48
    a = g.standard_normal((M, Nh)) * 4
    one = np.ones((M, Nh))
    y_pos = oracle.epilogue(oracle.interleave_gate_up(a, one), act=1)
    y_neg = oracle.epilogue(oracle.interleave_gate_up(-a, one), act=1)
    assert np.allclose(y_pos - y_neg, a, rtol=1e-12, atol=1e-15), "silu antisymmetry"
    big = oracle.epilogue(oracle.interleave_gate_up(np.full((1, 16), 40.0), np.full((1, 16), 3.0)), act=1)
    assert np.all(big == 120.0), "silu(40) * 3"
    neg = oracle.epilogue(oracle.interleave_gate_up(np.full((1, 16), -40.0), np.full((1, 16), 3.0)), act=1)
    assert np.all(np.abs(neg) < 1e-15) and np.all(neg < 0), "silu(-40)"
    zero = oracle.epilogue(oracle.interleave_gate_up(np.zeros((1, 16)), np.full((1, 16), 7.0)), act=1)
    assert np.all(zero == 0.0), "silu(0)"
    # the layout: each output column reads its own gate and up column
    gate = np.arange(Nh, dtype=np.float64)[None, :] * 0.01
    up = 1.0 + np.arange(Nh, dtype=np.float64)[None, :]
    h = oracle.interleave_gate_up(gate, up)
    assert h[0, 0] == gate[0, 0] and h[0, 15] == gate[0, 15] and h[0, 16] == up[0, 0]
    assert h[0, 31] == up[0, 15] and h[0, 32] == gate[0, 16] and h[0, 48] == up[0, 16]
    y = oracle.epilogue(h, act=1)
    want = gate / (1.0 + np.exp(-gate)) * up
    assert np.allclose(y, want, rtol=1e-15), "gate/up pairing"
    # bias: small integers, exact in binary16 and binary64
    b = _f16(g.integers(-8, 9, 2 * Nh).astype(np.float64))
    hi = g.integers(-100, 100, (M, 2 * Nh)).astype(np.float64)
    hb = oracle.epilogue(hi, bias_bits=b)
    assert np.array_equal(hb - hi, np.broadcast_to(b.view(np.float16).astype(np.float64), hi.shape)), "bias add"
    assert np.array_equal(oracle.epilogue(hi, bias_bits=b, act=1), oracle.epilogue(hb, act=1))


def pin_zero_when_z_equals_q():
    M, K, N = 3, 256, 32
    g = _rng(400)
    x = _f16(g.standard_normal((M, K)))
    z = g.integers(0, 16, (K // 128, N), dtype=np.uint8)
    q = np.repeat(z, 128, axis=0)
    s = _f16(g.uniform(0.002, 0.02, (K // 128, N)))
    y = oracle.gemm(x, q, z, s)
    assert np.all(y == 0.0), "z == q must give y == 0"


def pin_scale_doubling():
    x, q, z, s = _rand_case(500, 3, 256, 32)
    s2 = _f16(s.view(np.float16).astype(np.float64) * 2)
    assert np.array_equal(oracle.gemm(x, q, z, s2), 2 * oracle.gemm(x, q, z, s))


def pin_dequant_is_identity_gemm():
    _, q, z, s = _rand_case(600, 1, 256, 32)
    eye = np.full((256, 256), 0, np.uint16)
    eye[np.arange(256), np.arange(256)] = ONE_F16
    assert np.array_equal(oracle.dequant(q, z, s), oracle.gemm(eye, q, z, s))


def pin_column_sample():
    x, q, z, s = _rand_case(700, 2, 256, 64)
    cols = np.array([63, 0, 17, 31, 32], np.int64)
    full = oracle.gemm(x, q, z, s)
    assert np.array_equal(oracle.gemm(x, q, z, s, cols=cols), full[:, cols])


# ---------------------------------------------------------------- packing

def _locate(K, N, k, n):
    """Pack a tensor whose only non-zero element is q[k][n] = 5; return the
    (word, nibble) where the 5 lands."""
    q = np.zeros((K, N), np.uint8)
    q[k, n] = 5
    z = np.zeros((K // 128, N), np.uint8)
    s = np.zeros((K // 128, N), np.uint16)
    pw, _, _ = oracle.pack(q, z, s)
    nz = np.nonzero(pw)[0]
    assert nz.size == 1, "one element must land in exactly one word"
    w = int(pw[nz[0]])
    slots = [i for i in range(8) if (w >> (4 * i)) & 15]
    assert len(slots) == 1 and (w >> (4 * slots[0])) & 15 == 5
    return int(nz[0]), slots[0]


# (k, n) -> (word, nibble) for K = 256, N = 32, worked out by hand from the
# layout's prose definition: unit (n-tile, k-group) of 64 lanes x 4 words,
# lane = 16*(k%32 // 8) + n%16, word in lane = k%128 // 32, nibble slot of
# element e = k%8 is e/2 for even e and 4 + e/2 for odd e.
PACK_POSITIONS = {
    (0, 0): (0, 0),
    (1, 0): (0, 4),
    (2, 0): (0, 1),
    (7, 0): (0, 7),
    (6, 0): (0, 3),
    (8, 0): (64, 0),
    (32, 0): (1, 0),
    (127, 15): (255, 7),
    (128, 0): (256, 0),
    (0, 16): (512, 0),
    (200, 17): (838, 0),
    (45, 3): (4 * (16 * 1 + 3) + 1, 6),   # r=45: j=1, g=1, e=5 -> slot 6
}


def pin_pack_positions():
    for (k, n), want in PACK_POSITIONS.items():
        assert _locate(256, 32, k, n) == want, "packed position of q[%d][%d]" % (k, n)
    # zero point of (kg=1, n=17): word 3*2 + 0, nibble 1; scale: half 3*16 + 1
    K, N = 256, 32
    q = np.zeros((K, N), np.uint8)
    z = np.zeros((2, N), np.uint8)
    s = np.zeros((2, N), np.uint16)
    z[1, 17] = 9
    s[1, 17] = 0x1234
    _, pz, ps = oracle.pack(q, z, s)
    assert pz[6] == 9 << 4 and np.count_nonzero(pz) == 1
    assert ps[49] == 0x1234 and np.count_nonzero(ps) == 1


def pin_pack_bijection():
    """Index-encoded tensors: tensor b holds nibble b of each element's flat
    index; unpacking slot by slot recovers the source index of every slot,
    which must cover each of the K*N elements exactly once."""
    K, N = 256, 48
    flat = np.arange(K * N, dtype=np.int64).reshape(K, N)
    z = np.zeros((K // 128, N), np.uint8)
    s = np.zeros((K // 128, N), np.uint16)
    src = np.zeros(K * N, np.int64)
    for b in range(4):
        q = ((flat >> (4 * b)) & 15).astype(np.uint8)
        pw, _, _ = oracle.pack(q, z, s)
        nib = np.stack([(pw >> (4 * i)) & 15 for i in range(8)], axis=1).reshape(-1)
        src |= nib.astype(np.int64) << (4 * b)
    assert np.array_equal(np.sort(src), np.arange(K * N)), "layout is not a permutation"


ALL_PINS = [
    pin_f16_decode_all,
    pin_f16_encode,
    pin_integer_case,
    pin_closed_form,
    pin_exact_fraction,
    pin_grouped_exact_fraction,
    pin_epilogue_invariants,
    pin_zero_when_z_equals_q,
    pin_scale_doubling,
    pin_dequant_is_identity_gemm,
    pin_column_sample,
    pin_pack_positions,
    pin_pack_bijection,
]
