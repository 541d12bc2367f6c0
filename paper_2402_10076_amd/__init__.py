"""Python binding of libquick.so, the gfx950 W4A16 GEMM library.

Argument marshalling only: every step of the GEMM runs in the library's HIP
kernels and the offline pack runs in its host C++ code.  PyTorch provides the
device memory and the stream.  There is no fallback: if the library is not
built, importing the binding's functions raises.

Entry points mirror include/quick.h:

* ``packed_sizes(K, N, group=128)``
* ``pack_weights(q, z, s_bits, group=128)`` -> (packed, scales, zeros) numpy
* ``unpack_weights(packed, scales, zeros, K, N, group=128)``
* ``w4a16_gemm(x, packed, scales, zeros, N, y=None, group=128, ...)``
* ``select_config(M, N, K)``, ``workspace_bytes(M, N, K, cfg=None)``
* ``grouped_gemm(x, offsets, packed, scales, zeros, N, rows=None, ...)``
  (include/quick_grouped.h), ``pack_experts(experts)``
* ``gemm_fused`` / ``grouped_gemm_fused`` with a bias and the gated SiLU
  (include/quick_fused.h), ``interleave_gate_up(gate, up)``
"""
from __future__ import annotations

import ctypes
import os
import threading

# torch first: its HIP runtime (soname libamdhip64.so.7) is then the one
# libquick.so binds to, so the process has a single HIP runtime.
import torch  # noqa: E402
import numpy as np  # noqa: E402

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libquick.so")

QUICK_OK = 0
QUICK_ERR_INVALID_ARG = 1
QUICK_ERR_SHAPE = 2
QUICK_ERR_UNSUPPORTED = 3
QUICK_ERR_RANGE = 4
QUICK_ERR_ALIGNMENT = 5
QUICK_ERR_HIP = 6
QUICK_ERR_WORKSPACE = 7
QUICK_ERR_IO = 8
QUICK_ERR_CAPTURE = 9

VARIANT_AUTO = 0
VARIANT_STREAM = 1
VARIANT_TILED = 2
VARIANT_STREAMK = 3
VARIANT_KSTREAM = 5
VARIANT_TILED32 = 6
VARIANT_STREAMK32 = 7

# torch device type of every tensor whose address goes to the library (the
# CPU tests of the argument checks substitute "meta")
_DEVICE_TYPE = "cuda"

# leading workspace bytes that hold arrival counters (stream-K, sliced) (QUICK_WORKSPACE_COUNTER_BYTES)
WS_COUNTER_BYTES = 16384
# bytes of the per-GPU scratch array of quick_w4a16_gemm_noalloc (QUICK_SCRATCH_BYTES)
SCRATCH_BYTES = 80 << 20

_lock = threading.Lock()
_lib = None


class QuickError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        name = _lib.quick_status_string(int(status)).decode() if _lib is not None else "?"
        super().__init__("%s: %s (status %d)" % (what, name, status))


class QuickConfig(ctypes.Structure):
    _fields_ = [("variant", ctypes.c_int), ("split_k", ctypes.c_int),
                ("tile_m", ctypes.c_int), ("tile_n", ctypes.c_int)]

    def as_dict(self):
        return {f: getattr(self, f) for f, _ in self._fields_}


class QuickEpilogue(ctypes.Structure):
    _fields_ = [("bias", ctypes.c_void_p), ("activation", ctypes.c_int)]


ACT_NONE = 0
ACT_SILU_GATE = 1


def lib():
    """The loaded library (raises if it has not been built)."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                raise ImportError("libquick.so is not built (run __graft_entry__.build() or "
                                  "python -m paper_2402_10076_amd.build)")
            L = ctypes.CDLL(LIB_PATH)
            P, I64, SZ, I = ctypes.c_void_p, ctypes.c_int64, ctypes.c_size_t, ctypes.c_int
            L.quick_status_string.argtypes = [I]
            L.quick_status_string.restype = ctypes.c_char_p
            L.quick_pack_format_version.argtypes = []
            L.quick_pack_format_version.restype = I
            L.quick_packed_sizes.argtypes = [I64, I64, I64, ctypes.POINTER(SZ), ctypes.POINTER(SZ),
                                             ctypes.POINTER(SZ)]
            L.quick_packed_sizes.restype = I
            L.quick_pack_weights.argtypes = [P, P, P, I64, I64, I64, P, P, P]
            L.quick_pack_weights.restype = I
            L.quick_unpack_weights.argtypes = [P, P, P, I64, I64, I64, P, P, P]
            L.quick_unpack_weights.restype = I
            L.quick_w4a16_gemm.argtypes = [P, P, P, P, P, I64, I64, I64, I64, P]
            L.quick_w4a16_gemm.restype = I
            L.quick_w4a16_gemm_ex.argtypes = [P, P, P, P, P, I64, I64, I64, I64, P,
                                              ctypes.POINTER(QuickConfig), P, SZ]
            L.quick_w4a16_gemm_ex.restype = I
            L.quick_w4a16_gemm_noalloc.argtypes = [P, P, P, P, P, I64, I64, I64, I64, P]
            L.quick_w4a16_gemm_noalloc.restype = I
            L.quick_workspace_bytes.argtypes = [I64, I64, I64, ctypes.POINTER(QuickConfig)]
            L.quick_workspace_bytes.restype = SZ
            L.quick_select_config.argtypes = [I64, I64, I64, ctypes.POINTER(QuickConfig)]
            L.quick_select_config.restype = I
            L.quick_tune.argtypes = [P, P, P, P, P, I64, I64, I64, I64, P, ctypes.POINTER(QuickConfig)]
            L.quick_tune.restype = I
            L.quick_tune_table_save.argtypes = [ctypes.c_char_p]
            L.quick_tune_table_save.restype = I
            L.quick_tune_table_load.argtypes = [ctypes.c_char_p]
            L.quick_tune_table_load.restype = I
            L.quick_tune_table_size.argtypes = []
            L.quick_tune_table_size.restype = I
            L.quick_tune_table_clear.argtypes = []
            L.quick_tune_table_clear.restype = None
            L.quick_ablation_gemm.argtypes = [P, P, P, P, P, I64, I64, I64, I, P]
            L.quick_ablation_gemm.restype = I
            L.quick_w4a16_grouped_gemm.argtypes = [P, P, P, P, P, P, P, I64, I64, I64, I64, I64, I64, P]
            L.quick_w4a16_grouped_gemm.restype = I
            L.quick_w4a16_grouped_gemm_ex.argtypes = [P, P, P, P, P, P, P, I64, I64, I64, I64, I64, I64, P,
                                                      ctypes.POINTER(QuickConfig), P, SZ]
            L.quick_w4a16_grouped_gemm_ex.restype = I
            L.quick_grouped_workspace_bytes.argtypes = [I64, I64, I64, I64, ctypes.POINTER(QuickConfig)]
            L.quick_grouped_workspace_bytes.restype = SZ
            L.quick_grouped_select_config.argtypes = [I64, I64, I64, I64, ctypes.POINTER(QuickConfig)]
            L.quick_grouped_select_config.restype = I
            EP = ctypes.POINTER(QuickEpilogue)
            L.quick_w4a16_gemm_fused.argtypes = [P, P, P, P, P, I64, I64, I64, I64, P, EP,
                                                 ctypes.POINTER(QuickConfig), P, SZ]
            L.quick_w4a16_gemm_fused.restype = I
            L.quick_w4a16_grouped_gemm_fused.argtypes = [P, P, P, P, P, P, P, I64, I64, I64, I64, I64, I64, P, EP,
                                                         ctypes.POINTER(QuickConfig), P, SZ]
            L.quick_w4a16_grouped_gemm_fused.restype = I
            L.quick_fused_workspace_bytes.argtypes = [I64, I64, I64, ctypes.POINTER(QuickConfig), EP]
            L.quick_fused_workspace_bytes.restype = SZ
            L.quick_grouped_fused_workspace_bytes.argtypes = [I64, I64, I64, I64, ctypes.POINTER(QuickConfig), EP]
            L.quick_grouped_fused_workspace_bytes.restype = SZ
            L.quick_interleave_gate_up.argtypes = [P, P, P, P, P, P, I64, I64, I64, P, P, P]
            L.quick_interleave_gate_up.restype = I
            _lib = L
    return _lib


def status_string(status: int) -> str:
    return lib().quick_status_string(int(status)).decode()


def _check(st: int, what: str):
    if st != QUICK_OK:
        raise QuickError(st, what)


def _np_ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def pack_format_version() -> int:
    return lib().quick_pack_format_version()


def packed_sizes(K: int, N: int, group: int = 128):
    a, b, c = ctypes.c_size_t(), ctypes.c_size_t(), ctypes.c_size_t()
    _check(lib().quick_packed_sizes(K, N, group, ctypes.byref(a), ctypes.byref(b), ctypes.byref(c)),
           "quick_packed_sizes")
    return a.value, b.value, c.value


def pack_weights(q, z, s_bits, group: int = 128):
    """Offline reorder on the host.  q [K][N] uint8, z [K/g][N] uint8, s_bits
    [K/g][N] uint16 (binary16).  Returns numpy (packed u32, scales u16,
    zeros u32)."""
    q = np.ascontiguousarray(q, np.uint8)
    z = np.ascontiguousarray(z, np.uint8)
    s = np.ascontiguousarray(s_bits, np.uint16)
    K, N = q.shape
    if z.shape != (K // group, N) or s.shape != (K // group, N):
        raise QuickError(QUICK_ERR_SHAPE, "pack_weights: z and s must be [K/group][N]")
    wb, zb, sb = packed_sizes(K, N, group)
    pw = np.empty(wb // 4, np.uint32)
    ps = np.empty(sb // 2, np.uint16)
    pz = np.empty(zb // 4, np.uint32)
    _check(lib().quick_pack_weights(_np_ptr(q), _np_ptr(z), _np_ptr(s), K, N, group,
                                    _np_ptr(pw), _np_ptr(ps), _np_ptr(pz)), "quick_pack_weights")
    return pw, ps, pz


def unpack_weights(packed, scales, zeros, K: int, N: int, group: int = 128):
    pw = np.ascontiguousarray(packed, np.uint32)
    ps = np.ascontiguousarray(scales, np.uint16)
    pz = np.ascontiguousarray(zeros, np.uint32)
    wb, zb, sb = packed_sizes(K, N, group)
    if pw.nbytes != wb or ps.nbytes != sb or pz.nbytes != zb:
        raise QuickError(QUICK_ERR_SHAPE, "unpack_weights: buffer sizes do not match K, N")
    q = np.empty((K, N), np.uint8)
    z = np.empty((K // group, N), np.uint8)
    s = np.empty((K // group, N), np.uint16)
    _check(lib().quick_unpack_weights(_np_ptr(pw), _np_ptr(ps), _np_ptr(pz), K, N, group,
                                      _np_ptr(q), _np_ptr(z), _np_ptr(s)), "quick_unpack_weights")
    return q, z, s


def to_device(packed, scales, zeros, device="cuda"):
    """Copy host packed buffers into device tensors (int32 / int16 / int32)."""
    return (torch.from_numpy(np.ascontiguousarray(packed).view(np.int32)).to(device),
            torch.from_numpy(np.ascontiguousarray(scales).view(np.int16)).to(device),
            torch.from_numpy(np.ascontiguousarray(zeros).view(np.int32)).to(device))


def make_config(variant=0, split_k=0, tile_m=0, tile_n=0) -> QuickConfig:
    return QuickConfig(variant, split_k, tile_m, tile_n)


def select_config(M: int, N: int, K: int) -> dict:
    c = QuickConfig()
    _check(lib().quick_select_config(M, N, K, ctypes.byref(c)), "quick_select_config")
    return c.as_dict()


def workspace_bytes(M: int, N: int, K: int, cfg: QuickConfig | None = None) -> int:
    return int(lib().quick_workspace_bytes(M, N, K, ctypes.byref(cfg) if cfg is not None else None))


def _dptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)


def _nbytes(t: torch.Tensor) -> int:
    return t.numel() * t.element_size()


def _dev(what: str, name: str, t, ref: torch.Tensor, dtype=None, nbytes: int | None = None,
         shape: tuple | None = None):
    """Check that ``t`` is a contiguous tensor on ``ref``'s GPU (and of the
    given dtype, shape and minimum byte size) before its address is passed to
    the library: the kernels size their buffer descriptors from the shape
    arguments, so a host tensor or a short buffer would fault instead of
    being reported."""
    if not isinstance(t, torch.Tensor):
        raise QuickError(QUICK_ERR_INVALID_ARG, "%s: %s must be a torch tensor" % (what, name))
    if t.device.type != _DEVICE_TYPE or t.device != ref.device:
        raise QuickError(QUICK_ERR_INVALID_ARG, "%s: %s must be on %s, not %s" % (what, name, ref.device, t.device))
    if not t.is_contiguous():
        raise QuickError(QUICK_ERR_INVALID_ARG, "%s: %s must be contiguous" % (what, name))
    if dtype is not None and t.dtype != dtype:
        raise QuickError(QUICK_ERR_INVALID_ARG, "%s: %s must be %s, not %s" % (what, name, dtype, t.dtype))
    if shape is not None and tuple(t.shape) != tuple(shape):
        raise QuickError(QUICK_ERR_INVALID_ARG, "%s: %s must have shape %s, not %s" % (
            what, name, tuple(shape), tuple(t.shape)))
    if nbytes is not None and _nbytes(t) < nbytes:
        raise QuickError(QUICK_ERR_SHAPE, "%s: %s holds %d bytes, needs %d" % (what, name, _nbytes(t), nbytes))


def _check_x(what: str, x, rows_name: str = "M"):
    if not isinstance(x, torch.Tensor) or x.device.type != _DEVICE_TYPE:
        raise QuickError(QUICK_ERR_INVALID_ARG, "%s: x must be a tensor on the GPU" % what)
    if x.dtype != torch.float16 or x.dim() != 2 or not x.is_contiguous():
        raise QuickError(QUICK_ERR_INVALID_ARG,
                         "%s: x must be a contiguous [%s][K] float16 tensor" % (what, rows_name))


def _weight_bytes(what: str, K: int, N: int, group: int):
    """Byte sizes (packed, scales, zeros) of one K x N weight matrix (the
    quick_packed_sizes formulas: K*N/2, K*N/64, K*N/256)."""
    if group != 128:
        raise QuickError(QUICK_ERR_UNSUPPORTED, "%s: group must be 128" % what)
    if K <= 0 or N <= 0 or K % 128 or N % 16:
        raise QuickError(QUICK_ERR_SHAPE, "%s: need K %% 128 == 0 and N %% 16 == 0 (K=%d, N=%d)" % (what, K, N))
    return K * N // 2, K * N // 64, K * N // 256


def _check_weights(what: str, x, packed, scales, zeros, K: int, N: int, group: int, experts: int = 1):
    wb, sb, zb = _weight_bytes(what, K, N, group)
    _dev(what, "packed", packed, x, nbytes=wb * experts)
    _dev(what, "scales", scales, x, nbytes=sb * experts)
    _dev(what, "zeros", zeros, x, nbytes=zb * experts)


def _out(what: str, y, x, rows: int, cols: int):
    if y is None:
        return torch.empty((rows, cols), dtype=torch.float16, device=x.device)
    _dev(what, "y", y, x, dtype=torch.float16, shape=(rows, cols))
    return y


def _ws(what: str, workspace, x):
    if workspace is None:
        return 0
    _dev(what, "workspace", workspace, x)
    return _nbytes(workspace)


def _stream(stream, x):
    st = stream if stream is not None else torch.cuda.current_stream(x.device)
    return ctypes.c_void_p(st.cuda_stream)


def w4a16_gemm(x: torch.Tensor, packed: torch.Tensor, scales: torch.Tensor, zeros: torch.Tensor,
               N: int, y: torch.Tensor | None = None, group: int = 128,
               cfg: QuickConfig | None = None, workspace: torch.Tensor | None = None,
               stream=None) -> torch.Tensor:
    """y = x . W on the GPU.  x: [M][K] float16 (contiguous, on the device);
    packed/scales/zeros: device tensors from ``to_device``.  Runs on torch's
    current stream unless ``stream`` (a torch.cuda.Stream) is given."""
    what = "w4a16_gemm"
    _check_x(what, x)
    M, K = x.shape
    _check_weights(what, x, packed, scales, zeros, K, N, group)
    y = _out(what, y, x, M, N)
    wsb = _ws(what, workspace, x)
    hs = _stream(stream, x)
    if cfg is None and workspace is None:
        rc = lib().quick_w4a16_gemm(_dptr(x), _dptr(packed), _dptr(scales), _dptr(zeros), _dptr(y),
                                    M, N, K, group, hs)
    else:
        rc = lib().quick_w4a16_gemm_ex(_dptr(x), _dptr(packed), _dptr(scales), _dptr(zeros), _dptr(y),
                                       M, N, K, group, hs,
                                       ctypes.byref(cfg) if cfg is not None else None,
                                       _dptr(workspace), wsb)
    _check(rc, "quick_w4a16_gemm")
    return y


def w4a16_gemm_noalloc(x: torch.Tensor, packed: torch.Tensor, scales: torch.Tensor, zeros: torch.Tensor,
                       N: int, y: torch.Tensor, group: int = 128, stream=None) -> torch.Tensor:
    """quick_w4a16_gemm_noalloc: y = x . W with the library's fixed per-GPU
    scratch array as workspace (no allocation in the call; y must be given).
    Calls that may overlap on one GPU race on that array."""
    what = "w4a16_gemm_noalloc"
    _check_x(what, x)
    M, K = x.shape
    _check_weights(what, x, packed, scales, zeros, K, N, group)
    if y is None:
        raise QuickError(QUICK_ERR_INVALID_ARG, "%s: y must be given (the call allocates nothing)" % what)
    y = _out(what, y, x, M, N)
    hs = _stream(stream, x)
    _check(lib().quick_w4a16_gemm_noalloc(_dptr(x), _dptr(packed), _dptr(scales), _dptr(zeros), _dptr(y),
                                          M, N, K, group, hs), "quick_w4a16_gemm_noalloc")
    return y


def tune(x: torch.Tensor, packed: torch.Tensor, scales: torch.Tensor, zeros: torch.Tensor, N: int,
         y: torch.Tensor | None = None, group: int = 128, stream=None) -> dict:
    """Time every configuration for this shape on these buffers and record the
    fastest in the library's tune table (quick_tune); returns it."""
    what = "tune"
    _check_x(what, x)
    M, K = x.shape
    _check_weights(what, x, packed, scales, zeros, K, N, group)
    y = _out(what, y, x, M, N)
    hs = _stream(stream, x)
    c = QuickConfig()
    _check(lib().quick_tune(_dptr(x), _dptr(packed), _dptr(scales), _dptr(zeros), _dptr(y), M, N, K, group,
                            hs, ctypes.byref(c)), "quick_tune")
    return c.as_dict()


def ablation_gemm(x: torch.Tensor, packed: torch.Tensor, scales: torch.Tensor, zeros: torch.Tensor,
                  N: int, mode: int, y: torch.Tensor | None = None) -> torch.Tensor:
    """quick_ablation_gemm: mode 0 direct-to-register (the method), 1 / 2
    write-back through LDS with padded / unpadded rows."""
    what = "ablation_gemm"
    _check_x(what, x)
    M, K = x.shape
    _check_weights(what, x, packed, scales, zeros, K, N, 128)
    y = _out(what, y, x, M, N)
    hs = _stream(None, x)
    _check(lib().quick_ablation_gemm(_dptr(x), _dptr(packed), _dptr(scales), _dptr(zeros), _dptr(y), M, N, K,
                                     mode, hs), "quick_ablation_gemm")
    return y


def pack_experts(experts, group: int = 128):
    """Pack E experts' (q, z, s_bits) and concatenate them into the back-to-back
    buffers quick_w4a16_grouped_gemm takes.  Returns (packed, scales, zeros) numpy."""
    parts = [pack_weights(q, z, s, group) for q, z, s in experts]
    return tuple(np.concatenate([p[i] for p in parts]) for i in range(3))


def grouped_select_config(R: int, E: int, N: int, K: int) -> dict:
    c = QuickConfig()
    _check(lib().quick_grouped_select_config(R, E, N, K, ctypes.byref(c)), "quick_grouped_select_config")
    return c.as_dict()


def grouped_workspace_bytes(R: int, E: int, N: int, K: int, cfg: QuickConfig | None = None) -> int:
    return int(lib().quick_grouped_workspace_bytes(R, E, N, K, ctypes.byref(cfg) if cfg is not None else None))


def _grouped_args(what, x, offsets, rows, R, packed, scales, zeros, N, group):
    """Validated (T, K, E, R) of a grouped call."""
    _check_x(what, x, "T")
    T, K = x.shape
    if not isinstance(offsets, torch.Tensor) or offsets.dim() != 1 or offsets.numel() < 2:
        raise QuickError(QUICK_ERR_INVALID_ARG, "%s: offsets must be an int32 vector of E+1 entries" % what)
    _dev(what, "offsets", offsets, x, dtype=torch.int32)
    E = offsets.numel() - 1
    if rows is not None:
        if not isinstance(rows, torch.Tensor) or rows.dim() != 1:
            raise QuickError(QUICK_ERR_INVALID_ARG, "%s: rows must be an int32 vector" % what)
        _dev(what, "rows", rows, x, dtype=torch.int32)
        if R is not None and R != rows.numel():
            raise QuickError(QUICK_ERR_SHAPE, "%s: R disagrees with rows" % what)
        R = rows.numel()
    elif R is None:
        R = T
    _check_weights(what, x, packed, scales, zeros, K, N, group, experts=E)
    return T, K, E, R


def grouped_gemm(x: torch.Tensor, offsets: torch.Tensor, packed: torch.Tensor, scales: torch.Tensor,
                 zeros: torch.Tensor, N: int, rows: torch.Tensor | None = None, R: int | None = None,
                 y: torch.Tensor | None = None, group: int = 128, cfg: QuickConfig | None = None,
                 workspace: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """Grouped (mixture-of-experts) GEMM, quick_w4a16_grouped_gemm:
    y[r] = x[rows[r]] . W_e for offsets[e] <= r < offsets[e+1].

    x: [T][K] float16; offsets: int32 [E+1] on the device; rows: int32 [R] on
    the device, or None (row r reads x[r]; R defaults to T); packed / scales /
    zeros: the experts' buffers back to back (``pack_experts`` + ``to_device``)."""
    what = "grouped_gemm"
    T, K, E, R = _grouped_args(what, x, offsets, rows, R, packed, scales, zeros, N, group)
    y = _out(what, y, x, R, N)
    wsb = _ws(what, workspace, x)
    hs = _stream(stream, x)
    args = (_dptr(x), _dptr(rows), _dptr(offsets), _dptr(packed), _dptr(scales), _dptr(zeros), _dptr(y),
            T, R, E, N, K, group, hs)
    if cfg is None and workspace is None:
        rc = lib().quick_w4a16_grouped_gemm(*args)
    else:
        rc = lib().quick_w4a16_grouped_gemm_ex(*args, ctypes.byref(cfg) if cfg is not None else None,
                                               _dptr(workspace), wsb)
    _check(rc, "quick_w4a16_grouped_gemm")
    return y


def interleave_gate_up(gate, up, group: int = 128):
    """quick_interleave_gate_up: the column order the gated epilogue expects,
    from unpacked (q, z, s_bits) of the gate and up matrices ([K][Nh] each)."""
    qg, zg, sg = (np.ascontiguousarray(a) for a in gate)
    qu, zu, su = (np.ascontiguousarray(a) for a in up)
    K, Nh = qg.shape
    q = np.empty((K, 2 * Nh), np.uint8)
    z = np.empty((K // group, 2 * Nh), np.uint8)
    s = np.empty((K // group, 2 * Nh), np.uint16)
    _check(lib().quick_interleave_gate_up(_np_ptr(qg.astype(np.uint8)), _np_ptr(zg.astype(np.uint8)),
                                          _np_ptr(sg.astype(np.uint16)), _np_ptr(qu.astype(np.uint8)),
                                          _np_ptr(zu.astype(np.uint8)), _np_ptr(su.astype(np.uint16)),
                                          K, Nh, group, _np_ptr(q), _np_ptr(z), _np_ptr(s)),
           "quick_interleave_gate_up")
    return q, z, s


def _epi(bias, activation):
    return QuickEpilogue(ctypes.c_void_p(bias.data_ptr()) if bias is not None else None, int(activation))


def fused_workspace_bytes(M, N, K, cfg=None, bias=None, activation=0) -> int:
    e = _epi(bias, activation)
    return int(lib().quick_fused_workspace_bytes(M, N, K, ctypes.byref(cfg) if cfg is not None else None,
                                                 ctypes.byref(e)))


def _check_bias(what, bias, x, n):
    if bias is not None:
        _dev(what, "bias", bias, x, dtype=torch.float16, nbytes=2 * n)


def gemm_fused(x: torch.Tensor, packed: torch.Tensor, scales: torch.Tensor, zeros: torch.Tensor, N: int,
               bias: torch.Tensor | None = None, activation: int = ACT_NONE, y: torch.Tensor | None = None,
               group: int = 128, cfg: QuickConfig | None = None, workspace: torch.Tensor | None = None,
               stream=None) -> torch.Tensor:
    """quick_w4a16_gemm_fused: y = epilogue(x . W + bias); ``activation`` =
    ACT_SILU_GATE gives the [M][N/2] gated SiLU of interleaved gate/up tiles."""
    what = "gemm_fused"
    _check_x(what, x)
    M, K = x.shape
    _check_weights(what, x, packed, scales, zeros, K, N, group)
    _check_bias(what, bias, x, N)
    y = _out(what, y, x, M, N // 2 if activation == ACT_SILU_GATE else N)
    wsb = _ws(what, workspace, x)
    hs = _stream(stream, x)
    e = _epi(bias, activation)
    _check(lib().quick_w4a16_gemm_fused(_dptr(x), _dptr(packed), _dptr(scales), _dptr(zeros), _dptr(y), M, N, K,
                                        group, hs, ctypes.byref(e),
                                        ctypes.byref(cfg) if cfg is not None else None, _dptr(workspace), wsb),
           "quick_w4a16_gemm_fused")
    return y


def grouped_gemm_fused(x: torch.Tensor, offsets: torch.Tensor, packed: torch.Tensor, scales: torch.Tensor,
                       zeros: torch.Tensor, N: int, rows: torch.Tensor | None = None, R: int | None = None,
                       bias: torch.Tensor | None = None, activation: int = ACT_NONE,
                       y: torch.Tensor | None = None, group: int = 128, cfg: QuickConfig | None = None,
                       workspace: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """quick_w4a16_grouped_gemm_fused: the grouped GEMM with the epilogue
    (bias [E][N] per expert)."""
    what = "grouped_gemm_fused"
    T, K, E, R = _grouped_args(what, x, offsets, rows, R, packed, scales, zeros, N, group)
    _check_bias(what, bias, x, E * N)
    y = _out(what, y, x, R, N // 2 if activation == ACT_SILU_GATE else N)
    wsb = _ws(what, workspace, x)
    hs = _stream(stream, x)
    e = _epi(bias, activation)
    _check(lib().quick_w4a16_grouped_gemm_fused(_dptr(x), _dptr(rows), _dptr(offsets), _dptr(packed),
                                                _dptr(scales), _dptr(zeros), _dptr(y), T, R, E, N, K, group,
                                                hs, ctypes.byref(e),
                                                ctypes.byref(cfg) if cfg is not None else None,
                                                _dptr(workspace), wsb),
           "quick_w4a16_grouped_gemm_fused")
    return y


def tune_table_save(path: str) -> None:
    _check(lib().quick_tune_table_save(os.fsencode(path)), "quick_tune_table_save")


def tune_table_load(path: str) -> None:
    _check(lib().quick_tune_table_load(os.fsencode(path)), "quick_tune_table_load")


def tune_table_size() -> int:
    return int(lib().quick_tune_table_size())


def tune_table_clear() -> None:
    lib().quick_tune_table_clear()


EXPORTED = (
    "quick_status_string", "quick_pack_format_version", "quick_packed_sizes", "quick_pack_weights",
    "quick_unpack_weights", "quick_w4a16_gemm", "quick_w4a16_gemm_ex", "quick_w4a16_gemm_noalloc",
    "quick_workspace_bytes",
    "quick_select_config", "quick_tune", "quick_tune_table_save", "quick_tune_table_load",
    "quick_tune_table_size", "quick_tune_table_clear", "quick_ablation_gemm",
    "quick_w4a16_grouped_gemm", "quick_w4a16_grouped_gemm_ex", "quick_grouped_workspace_bytes",
    "quick_grouped_select_config", "quick_w4a16_gemm_fused", "quick_w4a16_grouped_gemm_fused",
    "quick_fused_workspace_bytes", "quick_grouped_fused_workspace_bytes", "quick_interleave_gate_up",
)
