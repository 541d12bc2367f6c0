"""The binding's argument checks, on the CPU: every wrapper rejects a host
tensor, a tensor on another device, a non-contiguous or mistyped tensor and
a buffer shorter than the shape requires before it takes a stream or calls
into the library.  The library is replaced by a stub that records calls, and
"meta" tensors stand in for device tensors, so no kernel can be reached."""
import pytest
import torch

import paper_2402_10076_amd as Q


class _Stub:
    """Records every library entry point called; each returns QUICK_OK."""

    def __init__(self):
        self.calls = []

    def __getattr__(self, name):
        def f(*a):
            self.calls.append(name)
            return Q.QUICK_OK
        return f


class _Stream:
    cuda_stream = 0


@pytest.fixture
def stub(monkeypatch):
    s = _Stub()
    monkeypatch.setattr(Q, "lib", lambda: s)
    monkeypatch.setattr(Q, "_DEVICE_TYPE", "meta")
    return s


M, K, N = 4, 256, 32


def _dev(*shape, dtype=torch.int32):
    return torch.empty(shape, dtype=dtype, device="meta")


def _gemm_args():
    x = _dev(M, K, dtype=torch.float16)
    return x, _dev(K * N // 8), _dev(K * N // 128, dtype=torch.int16), _dev(K * N // 1024)


def _rejects(status, fn, *a, **kw):
    with pytest.raises(Q.QuickError) as e:
        fn(*a, **kw)
    assert e.value.status == status


def test_valid_call_reaches_library(stub):
    x, pw, ps, pz = _gemm_args()
    y = Q.w4a16_gemm(x, pw, ps, pz, N, stream=_Stream())
    assert tuple(y.shape) == (M, N) and stub.calls == ["quick_w4a16_gemm"]


@pytest.mark.parametrize("which", ["x", "packed", "scales", "zeros", "y", "workspace"])
def test_host_tensor_rejected(stub, which):
    x, pw, ps, pz = _gemm_args()
    args = dict(x=x, packed=pw, scales=ps, zeros=pz, y=_dev(M, N, dtype=torch.float16),
                workspace=_dev(1024))
    args[which] = torch.zeros(tuple(args[which].shape), dtype=args[which].dtype)   # on the host
    _rejects(Q.QUICK_ERR_INVALID_ARG, Q.w4a16_gemm, args["x"], args["packed"], args["scales"], args["zeros"], N,
             y=args["y"], workspace=args["workspace"], stream=_Stream())
    assert stub.calls == []


@pytest.mark.parametrize("which,nbytes", [("packed", K * N // 2 - 4), ("scales", K * N // 64 - 2),
                                          ("zeros", K * N // 256 - 4)])
def test_short_weight_buffer_rejected(stub, which, nbytes):
    x, pw, ps, pz = _gemm_args()
    bufs = dict(packed=pw, scales=ps, zeros=pz)
    t = bufs[which]
    bufs[which] = _dev(nbytes // t.element_size(), dtype=t.dtype)
    _rejects(Q.QUICK_ERR_SHAPE, Q.w4a16_gemm, x, bufs["packed"], bufs["scales"], bufs["zeros"], N, stream=_Stream())
    _rejects(Q.QUICK_ERR_SHAPE, Q.tune, x, bufs["packed"], bufs["scales"], bufs["zeros"], N, stream=_Stream())
    _rejects(Q.QUICK_ERR_SHAPE, Q.ablation_gemm, x, bufs["packed"], bufs["scales"], bufs["zeros"], N, 0)
    assert stub.calls == []


def test_wrong_output_and_layout_rejected(stub):
    x, pw, ps, pz = _gemm_args()
    _rejects(Q.QUICK_ERR_INVALID_ARG, Q.w4a16_gemm, x, pw, ps, pz, N, y=_dev(M, N + 16, dtype=torch.float16),
             stream=_Stream())
    _rejects(Q.QUICK_ERR_INVALID_ARG, Q.w4a16_gemm, x, pw, ps, pz, N, y=_dev(M, N, dtype=torch.float32),
             stream=_Stream())
    _rejects(Q.QUICK_ERR_INVALID_ARG, Q.w4a16_gemm, x.t(), pw, ps, pz, N, stream=_Stream())
    _rejects(Q.QUICK_ERR_INVALID_ARG, Q.w4a16_gemm, _dev(M, K, dtype=torch.float32), pw, ps, pz, N, stream=_Stream())
    wide = _dev(K * N // 4)[::2]                      # enough elements, not contiguous
    _rejects(Q.QUICK_ERR_INVALID_ARG, Q.w4a16_gemm, x, wide, ps, pz, N, stream=_Stream())
    _rejects(Q.QUICK_ERR_SHAPE, Q.w4a16_gemm, x, pw, ps, pz, N + 8, stream=_Stream())   # N % 16
    _rejects(Q.QUICK_ERR_UNSUPPORTED, Q.w4a16_gemm, x, pw, ps, pz, N, group=64, stream=_Stream())
    assert stub.calls == []


def test_fused_checks(stub):
    x, pw, ps, pz = _gemm_args()
    _rejects(Q.QUICK_ERR_SHAPE, Q.gemm_fused, x, pw, ps, pz, N, bias=_dev(N - 4, dtype=torch.float16),
             stream=_Stream())
    _rejects(Q.QUICK_ERR_INVALID_ARG, Q.gemm_fused, x, pw, ps, pz, N, bias=_dev(N, dtype=torch.float32),
             stream=_Stream())
    _rejects(Q.QUICK_ERR_INVALID_ARG, Q.gemm_fused, x, pw, ps, pz, N, activation=Q.ACT_SILU_GATE,
             y=_dev(M, N, dtype=torch.float16), stream=_Stream())      # gated output has N/2 columns
    assert stub.calls == []
    y = Q.gemm_fused(x, pw, ps, pz, N, bias=_dev(N, dtype=torch.float16), activation=Q.ACT_SILU_GATE,
                     stream=_Stream())
    assert tuple(y.shape) == (M, N // 2) and stub.calls == ["quick_w4a16_gemm_fused"]


def test_grouped_checks(stub):
    E, T = 3, 10
    x = _dev(T, K, dtype=torch.float16)
    pw, ps, pz = _dev(E * K * N // 8), _dev(E * K * N // 128, dtype=torch.int16), _dev(E * K * N // 1024)
    off = _dev(E + 1)
    rows = _dev(12)
    _rejects(Q.QUICK_ERR_SHAPE, Q.grouped_gemm, x, off, pw[:-1], ps, pz, N, rows=rows, stream=_Stream())
    _rejects(Q.QUICK_ERR_INVALID_ARG, Q.grouped_gemm, x, _dev(E + 1, dtype=torch.int64), pw, ps, pz, N,
             stream=_Stream())
    _rejects(Q.QUICK_ERR_INVALID_ARG, Q.grouped_gemm, x, torch.zeros(E + 1, dtype=torch.int32), pw, ps, pz, N,
             stream=_Stream())
    _rejects(Q.QUICK_ERR_INVALID_ARG, Q.grouped_gemm, x, off, pw, ps, pz, N, rows=torch.zeros(12, dtype=torch.int32),
             stream=_Stream())
    _rejects(Q.QUICK_ERR_SHAPE, Q.grouped_gemm, x, off, pw, ps, pz, N, rows=rows, R=11, stream=_Stream())
    _rejects(Q.QUICK_ERR_SHAPE, Q.grouped_gemm_fused, x, off, pw, ps, pz, N, rows=rows,
             bias=_dev(E * N - 1, dtype=torch.float16), stream=_Stream())
    assert stub.calls == []
    y = Q.grouped_gemm(x, off, pw, ps, pz, N, rows=rows, stream=_Stream())
    assert tuple(y.shape) == (12, N) and stub.calls == ["quick_w4a16_grouped_gemm"]
