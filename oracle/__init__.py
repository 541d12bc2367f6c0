"""CPU oracle for the W4A16 GEMM -- TEST INFRASTRUCTURE ONLY.

Only the tests, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product path (the HIP library and
its Python binding) never touches it, and the two share no code.

The arithmetic lives in ``oracle.c`` (plain C, binary64):

* ``dequant``  -- W = (q - z) * s per group of 128 input channels
  (paper, Section 2.1 and Section 2.3).
* ``gemm``     -- y = x . W as a naive loop over k in ascending order.
* ``grouped_gemm`` (Python) -- the mixture-of-experts form: each expert's
  rows are ``gemm`` of its gathered token rows.
* ``epilogue`` / ``interleave_gate_up`` (Python) -- the fused output
  epilogue (bias, gated SiLU) and the gate/up column order it reads.
* ``pack``     -- the QPK16 offline reorder written as its element-wise
  definition (paper, Section 3.2 describes reordering the static weights
  offline to the matrix-instruction operand pattern and to the dequantizer's
  nibble order; the concrete layout is this project's gfx950 design).
* ``f16_to_f64`` / ``f64_to_f16`` -- binary16 decode and round-to-nearest-
  even encode written from the IEEE 754 format definition.

This module only marshals numpy arrays into that library.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lock = threading.Lock()
_lib = None


def build(force: bool = False) -> str:
    """Compile oracle.c into liboracle.so with gcc (no fast-math)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        cmd = ["gcc", "-O2", "-fopenmp", "-shared", "-fPIC", "-std=c11",
               "-Wall", "-Wextra", "-o", tmp, _SRC, "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB)
    return _LIB


def _bind(path: str):
    lib = ctypes.CDLL(path)
    P = ctypes.c_void_p
    I64 = ctypes.c_int64
    lib.oracle_f16_to_f64_array.argtypes = [P, I64, P]
    lib.oracle_f16_to_f64_array.restype = None
    lib.oracle_f64_to_f16_array.argtypes = [P, I64, P]
    lib.oracle_f64_to_f16_array.restype = None
    lib.oracle_dequant_f64.argtypes = [P, P, P, I64, I64, I64, P]
    lib.oracle_dequant_f64.restype = ctypes.c_int
    lib.oracle_gemm_f64.argtypes = [P, P, P, P, I64, I64, I64, I64, P, I64, P, ctypes.c_int]
    lib.oracle_gemm_f64.restype = ctypes.c_int
    lib.oracle_pack_qpk16.argtypes = [P, P, P, I64, I64, I64, P, P, P]
    lib.oracle_pack_qpk16.restype = ctypes.c_int
    lib.oracle_max_threads.argtypes = []
    lib.oracle_max_threads.restype = ctypes.c_int
    return lib


def _load():
    global _lib
    with _lock:
        if _lib is None:
            build()
            _lib = _bind(_LIB)
    return _lib


class use_library:
    """Context manager: route this module's calls to another build of
    oracle.c (used by the mutation tests that check the pins catch planted
    mistakes)."""

    def __init__(self, path: str):
        self.path = path

    def __enter__(self):
        global _lib
        _load()
        with _lock:
            self._saved = _lib
            _lib = _bind(self.path)
        return self

    def __exit__(self, *exc):
        global _lib
        with _lock:
            _lib = self._saved
        return False


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(np.asarray(a), dtype=dtype)


class OracleError(RuntimeError):
    pass


def f16_to_f64(bits) -> np.ndarray:
    """binary16 bit patterns (uint16) -> binary64 values."""
    b = _c(bits, np.uint16)
    out = np.empty(b.shape, np.float64)
    _load().oracle_f16_to_f64_array(_ptr(b), b.size, _ptr(out))
    return out


def f64_to_f16(values) -> np.ndarray:
    """binary64 values -> binary16 bit patterns, round to nearest, ties to even."""
    v = _c(values, np.float64)
    out = np.empty(v.shape, np.uint16)
    _load().oracle_f64_to_f16_array(_ptr(v), v.size, _ptr(out))
    return out


def dequant(q, z, s_bits, group: int = 128) -> np.ndarray:
    """W[k][n] = (q[k][n] - z[k//g][n]) * s[k//g][n] in binary64."""
    q = _c(q, np.uint8)
    z = _c(z, np.uint8)
    s = _c(s_bits, np.uint16)
    K, N = q.shape
    if z.shape != (K // group, N) or s.shape != (K // group, N):
        raise OracleError("z/s must be [K/group][N]")
    W = np.empty((K, N), np.float64)
    rc = _load().oracle_dequant_f64(_ptr(q), _ptr(z), _ptr(s), K, N, group, _ptr(W))
    if rc:
        raise OracleError("oracle_dequant_f64 failed with status %d" % rc)
    return W


def gemm(x_bits, q, z, s_bits, group: int = 128, cols=None, threads: int = 0) -> np.ndarray:
    """y = x . W in binary64, k ascending.  ``x_bits``: [M][K] binary16 bits.

    ``cols`` (optional) restricts the computation to those output columns;
    the result is then [M][len(cols)].
    """
    x = _c(x_bits, np.uint16)
    q = _c(q, np.uint8)
    z = _c(z, np.uint8)
    s = _c(s_bits, np.uint16)
    M, K = x.shape
    K2, N = q.shape
    if K2 != K:
        raise OracleError("x and q disagree on K")
    if z.shape != (K // group, N) or s.shape != (K // group, N):
        raise OracleError("z/s must be [K/group][N]")
    if cols is None:
        cp = None
        nc = N
        colarr = None
    else:
        colarr = _c(cols, np.int64)
        nc = colarr.size
        cp = _ptr(colarr)
    y = np.empty((M, nc), np.float64)
    rc = _load().oracle_gemm_f64(_ptr(x), _ptr(q), _ptr(z), _ptr(s), M, N, K, group,
                                 cp, nc, _ptr(y), int(threads))
    if rc:
        raise OracleError("oracle_gemm_f64 failed with status %d" % rc)
    return y


def grouped_gemm(x_bits, rows, offsets, experts, group: int = 128, cols=None, threads: int = 0) -> np.ndarray:
    """Mixture-of-experts form: routed row r is token row ``rows[r]`` of x
    (r itself when ``rows`` is None) multiplied by the weights of the expert
    e with offsets[e] <= r < offsets[e+1].  ``experts``: list of (q, z, s_bits).
    Each expert's block of rows is :func:`gemm` of its gathered token rows
    (the per-element definition is the dense GEMM's, Sections 2.1 and 2.3)."""
    x = _c(x_bits, np.uint16)
    off = np.asarray(offsets, np.int64)
    E = len(experts)
    if off.shape != (E + 1,) or off[0] != 0 or np.any(np.diff(off) < 0):
        raise OracleError("offsets must be non-decreasing [E+1] starting at 0")
    R = int(off[-1])
    r_tok = np.arange(R, dtype=np.int64) if rows is None else np.asarray(rows, np.int64)
    if r_tok.shape != (R,) or (R and (r_tok.min() < 0 or r_tok.max() >= x.shape[0])):
        raise OracleError("rows must be [R] token indices of x")
    N = experts[0][0].shape[1]
    nc = N if cols is None else len(cols)
    y = np.zeros((R, nc), np.float64)
    for e, (q, z, s) in enumerate(experts):
        lo, hi = int(off[e]), int(off[e + 1])
        if hi > lo:
            y[lo:hi] = gemm(x[r_tok[lo:hi]], q, z, s, group=group, cols=cols, threads=threads)
    return y


def epilogue(h, bias_bits=None, act: int = 0) -> np.ndarray:
    """Output epilogue of the fused GEMM in binary64: h + bias (bias as
    binary16 bits), then for act = 1 the gated SiLU of alternating 16-column
    gate / up tiles, y[m][16t + i] = silu(h[m][32t + i]) * h[m][32t + 16 + i],
    silu(a) = a / (1 + exp(-a))."""
    h = np.asarray(h, np.float64)
    if bias_bits is not None:
        h = h + f16_to_f64(bias_bits)[None, :]
    if act == 0:
        return h
    M, N = h.shape
    tiles = h.reshape(M, N // 32, 2, 16)
    gate, up = tiles[:, :, 0, :], tiles[:, :, 1, :]
    return (gate / (1.0 + np.exp(-gate)) * up).reshape(M, N // 2)


def interleave_gate_up(gate, up) -> np.ndarray:
    """Columns of two [R][Nh] arrays alternated in 16-column tiles: output
    column 32t + i is gate column 16t + i (i < 16), else up column 16t + i - 16."""
    g = np.asarray(gate)
    u = np.asarray(up)
    R, Nh = g.shape
    return np.stack([g.reshape(R, Nh // 16, 16), u.reshape(R, Nh // 16, 16)], axis=2).reshape(R, 2 * Nh)


def pack(q, z, s_bits, group: int = 128):
    """QPK16 layout, element-wise definition.  Returns (pw u32, pz u32, ps u16)."""
    q = _c(q, np.uint8)
    z = _c(z, np.uint8)
    s = _c(s_bits, np.uint16)
    K, N = q.shape
    pw = np.empty(K * N // 8, np.uint32)
    pz = np.empty(K * N // 1024, np.uint32)
    ps = np.empty(K * N // 128, np.uint16)
    rc = _load().oracle_pack_qpk16(_ptr(q), _ptr(z), _ptr(s), K, N, group,
                                   _ptr(pw), _ptr(pz), _ptr(ps))
    if rc:
        raise OracleError("oracle_pack_qpk16 failed with status %d" % rc)
    return pw, pz, ps


def max_threads() -> int:
    return int(_load().oracle_max_threads())
