"""ctypes binding of libmxattn (include/mxattn.h).

Argument marshalling only: every step of the hot path runs in the HIP
library.  PyTorch provides device memory and the current stream.  There is no
CPU fallback; if ``libmxattn.so`` is missing or cannot be loaded, every call
raises.
"""
from __future__ import annotations

import ctypes
import os
import threading

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libmxattn.so")

MODES = {"ocp_vanilla": 0, "uos": 1, "uos_pnq": 2, "uos_pnq_rot": 3}
AXIS_TOKENS, AXIS_HEAD_DIM = 2, 3
OK = 0

_lock = threading.Lock()
_lib = None


class MxattnError(RuntimeError):
    def __init__(self, status: int, where: str):
        L = lib()
        msg = L.mxattn_status_string(status).decode()
        detail = L.mxattn_last_error().decode()
        super().__init__(f"{where}: status {status} ({msg}){': ' + detail if detail else ''}")
        self.status = status


def lib() -> ctypes.CDLL:
    """Load libmxattn.so (built in-tree by ``python -m paper_2607_24377_amd.build``)."""
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(LIB_PATH):
                raise RuntimeError(
                    f"{LIB_PATH} is missing: build it with `python -m paper_2607_24377_amd.build`")
            L = ctypes.CDLL(LIB_PATH)
            P, I, I64, SZ = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64, ctypes.c_size_t
            L.mxattn_quantize.argtypes = [P, P, P, I, I, I64, I64, I64, I64, P]
            L.mxattn_quantize.restype = I
            D = ctypes.c_double
            L.mxattn_quantize_qmax.argtypes = [P, P, P, I, D, I64, I64, I64, I64, P]
            L.mxattn_quantize_qmax.restype = I
            L.mxattn_qmax_sse.argtypes = [P, I, P, I, P, I64, I64, I64, I64, P]
            L.mxattn_qmax_sse.restype = I
            F = ctypes.c_float
            L.mxattn_softmax_rows.argtypes = [P, P, P, I64, I64, I64, I64, I64, I64, I64, I64, P]
            L.mxattn_softmax_rows.restype = I
            L.mxattn_rowsum_diag.argtypes = [P, I64, I64, I64, I, F, P, P]
            L.mxattn_rowsum_diag.restype = I
            L.mxattn_attention_rowsum_diag.argtypes = [P, P, I64, I64, I64, I64, I64, I, F, P, P]
            L.mxattn_attention_rowsum_diag.restype = I
            L.mxattn_forward.argtypes = [P, P, P, P, I64, I64, I64, I64, I, P]
            L.mxattn_forward.restype = I
            L.mxattn_attend.argtypes = [P, P, P, P, P, P, P, I64, I64, I64, I64, I, P]
            L.mxattn_cross_forward.argtypes = [P, P, P, P, I64, I64, I64, I64, I64, I, P]
            L.mxattn_cross_forward.restype = I
            L.mxattn_cross_attend.argtypes = [P, P, P, P, P, P, P, I64, I64, I64, I64, I64, I, P]
            L.mxattn_cross_attend.restype = I
            L.mxattn_cross_attend_noalloc.argtypes = [P, P, P, P, P, P, P, I64, I64, I64, I64, I64, I, P]
            L.mxattn_cross_attend_noalloc.restype = I
            L.mxattn_attend.restype = I
            L.mxattn_codes_bytes.argtypes = [I, I64, I64, I64, I64]
            L.mxattn_codes_bytes.restype = SZ
            L.mxattn_scales_bytes.argtypes = [I, I64, I64, I64, I64]
            L.mxattn_scales_bytes.restype = SZ
            L.mxattn_kv_tile.argtypes = []
            L.mxattn_kv_tile.restype = I
            L.mxattn_query_tile.argtypes = []
            L.mxattn_query_tile.restype = I
            L.mxattn_status_string.argtypes = [I]
            L.mxattn_status_string.restype = ctypes.c_char_p
            L.mxattn_last_error.argtypes = []
            L.mxattn_last_error.restype = ctypes.c_char_p
            L.mxattn_release_workspace.argtypes = []
            L.mxattn_release_workspace.restype = I
            L.mxattn_version.argtypes = []
            L.mxattn_version.restype = I
            _lib = L
    return _lib


def _mode(mode) -> int:
    return MODES[mode] if isinstance(mode, str) else int(mode)


def _stream(stream) -> int:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _check(st: int, where: str):
    if st != OK:
        raise MxattnError(st, where)


def kv_tile() -> int:
    return lib().mxattn_kv_tile()


def query_tile() -> int:
    return lib().mxattn_query_tile()


def code_shapes(block_axis: int, B: int, H: int, N: int, d: int = 128):
    """Shapes of the codes and scales arrays of a [B, H, N, d] tensor."""
    if block_axis == AXIS_HEAD_DIM:
        return (B, H, N, d // 2), (B, H, N, d // 32)
    nb = (N + 31) // 32
    return (B, H, d, nb * 16), (B, H, d, nb)


def _bhnd(x: torch.Tensor):
    if x.dim() != 4:
        raise ValueError("expected a [B, H, N, d] tensor")
    if x.dtype != torch.bfloat16 or not x.is_cuda or not x.is_contiguous():
        raise ValueError("expected a contiguous bf16 CUDA tensor")
    return x.shape


def quantize(x: torch.Tensor, block_axis: int, mode, stream=None, codes=None, scales=None):
    """MXFP4-quantize bf16 x [B, H, N, d]; returns (codes, scales) uint8 tensors."""
    B, H, N, d = _bhnd(x)
    cs, ss = code_shapes(block_axis, B, H, N, d)
    if codes is None:
        codes = torch.empty(cs, dtype=torch.uint8, device=x.device)
    if scales is None:
        scales = torch.empty(ss, dtype=torch.uint8, device=x.device)
    st = lib().mxattn_quantize(x.data_ptr(), codes.data_ptr(), scales.data_ptr(), block_axis,
                               _mode(mode), B, H, N, d, _stream(stream))
    _check(st, "mxattn_quantize")
    return codes, scales


def quantize_qmax(x: torch.Tensor, block_axis: int, qmax: float, stream=None, codes=None, scales=None):
    """MXFP4-quantize bf16 x [B, H, N, d] with the ceil rule of boundary qmax."""
    B, H, N, d = _bhnd(x)
    cs, ss = code_shapes(block_axis, B, H, N, d)
    if codes is None:
        codes = torch.empty(cs, dtype=torch.uint8, device=x.device)
    if scales is None:
        scales = torch.empty(ss, dtype=torch.uint8, device=x.device)
    st = lib().mxattn_quantize_qmax(x.data_ptr(), codes.data_ptr(), scales.data_ptr(), block_axis,
                                    float(qmax), B, H, N, d, _stream(stream))
    _check(st, "mxattn_quantize_qmax")
    return codes, scales


def qmax_sse(x: torch.Tensor, block_axis: int, qs, stream=None, out=None):
    """Per-(batch, head) sum of squared MXFP4 errors of bf16 x [B, H, N, d] for
    each boundary in qs; returns a float64 device tensor [B*H, len(qs)]."""
    B, H, N, d = _bhnd(x)
    q = (ctypes.c_double * len(qs))(*[float(v) for v in qs])
    if out is None:
        out = torch.empty((B * H, len(qs)), dtype=torch.float64, device=x.device)
    st = lib().mxattn_qmax_sse(x.data_ptr(), block_axis, ctypes.cast(q, ctypes.c_void_p), len(qs),
                               out.data_ptr(), B, H, N, d, _stream(stream))
    _check(st, "mxattn_qmax_sse")
    return out


DIAG_FIELDS = ("rowsum", "mass", "zeroing", "saturation", "down", "up", "exact", "entropy")


def softmax_rows(q: torch.Tensor, k: torch.Tensor, row0: int = 0, rows: int | None = None, ld=None,
                 stream=None, out=None):
    """fp32 softmax(q k^T / sqrt(d)) for query rows [row0, row0 + rows) of
    every head: [B, H, rows, ld] (ld = Nkv rounded up to 4; entries past Nkv
    are left as allocated)."""
    B, H, Nq, d = _bhnd(q)
    Bk, Hk, Nkv, dk = _bhnd(k)
    if (Bk, Hk, dk) != (B, H, d):
        raise ValueError("k must be [B, H, Nkv, d] with q's B, H, d")
    rows = Nq - row0 if rows is None else rows
    ld = (Nkv + 3) // 4 * 4 if ld is None else ld
    if out is None:
        out = torch.empty((B, H, rows, ld), dtype=torch.float32, device=q.device)
    st = lib().mxattn_softmax_rows(q.data_ptr(), k.data_ptr(), out.data_ptr(), B, H, Nq, Nkv, d, row0,
                                   rows, ld, _stream(stream))
    _check(st, "mxattn_softmax_rows")
    return out


def rowsum_diag(p: torch.Tensor, N: int, mode, gamma: float = 1.0, stream=None, out=None):
    """Row-sum diagnostics of fp32 rows p [..., ld] (first N entries): [rows, 8]
    float64 in DIAG_FIELDS order."""
    if p.dtype != torch.float32 or not p.is_cuda or not p.is_contiguous():
        raise ValueError("expected a contiguous fp32 CUDA tensor")
    ld = p.shape[-1]
    rows = p.numel() // ld
    if out is None:
        out = torch.empty((rows, 8), dtype=torch.float64, device=p.device)
    st = lib().mxattn_rowsum_diag(p.data_ptr(), rows, N, ld, _mode(mode), float(gamma), out.data_ptr(),
                                  _stream(stream))
    _check(st, "mxattn_rowsum_diag")
    return out


def attention_rowsum_diag(q: torch.Tensor, k: torch.Tensor, mode, gamma: float = 1.0, stream=None,
                          out=None):
    """Row-sum diagnostics of every attention row: [B, H, Nq, 8] float64."""
    B, H, Nq, d = _bhnd(q)
    Bk, Hk, Nkv, dk = _bhnd(k)
    if (Bk, Hk, dk) != (B, H, d):
        raise ValueError("k must be [B, H, Nkv, d] with q's B, H, d")
    if out is None:
        out = torch.empty((B, H, Nq, 8), dtype=torch.float64, device=q.device)
    st = lib().mxattn_attention_rowsum_diag(q.data_ptr(), k.data_ptr(), B, H, Nq, Nkv, d, _mode(mode),
                                            float(gamma), out.data_ptr(), _stream(stream))
    _check(st, "mxattn_attention_rowsum_diag")
    return out


def forward(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, mode, out=None, stream=None):
    """MXFP4 attention forward of bf16 q, k, v [B, H, N, d]; returns bf16 out."""
    B, H, N, d = _bhnd(q)
    if _bhnd(k) != q.shape or _bhnd(v) != q.shape:
        raise ValueError("q, k, v must have the same shape")
    if out is None:
        out = torch.empty_like(q)
    st = lib().mxattn_forward(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(), B, H, N, d,
                              _mode(mode), _stream(stream))
    _check(st, "mxattn_forward")
    return out


def attend(qc, qs, kc, ks, vc, vs, N: int, mode, out=None, stream=None):
    """The fused kernel on quantized operands (library layouts); returns bf16 out."""
    B, H = qc.shape[0], qc.shape[1]
    d = qc.shape[3] * 2
    if out is None:
        out = torch.empty((B, H, N, d), dtype=torch.bfloat16, device=qc.device)
    st = lib().mxattn_attend(qc.data_ptr(), qs.data_ptr(), kc.data_ptr(), ks.data_ptr(),
                             vc.data_ptr(), vs.data_ptr(), out.data_ptr(), B, H, N, d, _mode(mode),
                             _stream(stream))
    _check(st, "mxattn_attend")
    return out


def cross_forward(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, mode, out=None, stream=None):
    """Attention of bf16 q [B, H, Nq, d] over k, v [B, H, Nkv, d]; returns bf16 out [B, H, Nq, d]."""
    B, H, Nq, d = _bhnd(q)
    Bk, Hk, Nkv, dk = _bhnd(k)
    if (Bk, Hk, dk) != (B, H, d) or _bhnd(v) != k.shape:
        raise ValueError("k and v must be [B, H, Nkv, d] with q's B, H, d")
    if out is None:
        out = torch.empty_like(q)
    st = lib().mxattn_cross_forward(q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(), B, H,
                                    Nq, Nkv, d, _mode(mode), _stream(stream))
    _check(st, "mxattn_cross_forward")
    return out


def cross_attend(qc, qs, kc, ks, vc, vs, Nq: int, Nkv: int, mode, out=None, stream=None):
    """The fused kernel on quantized operands with Nq queries and Nkv keys."""
    B, H = qc.shape[0], qc.shape[1]
    d = qc.shape[3] * 2
    if out is None:
        out = torch.empty((B, H, Nq, d), dtype=torch.bfloat16, device=qc.device)
    st = lib().mxattn_cross_attend(qc.data_ptr(), qs.data_ptr(), kc.data_ptr(), ks.data_ptr(),
                                   vc.data_ptr(), vs.data_ptr(), out.data_ptr(), B, H, Nq, Nkv, d,
                                   _mode(mode), _stream(stream))
    _check(st, "mxattn_cross_attend")
    return out


def bf16_from_bits(bits, device="cuda") -> torch.Tensor:
    """bf16 tensor from a numpy uint16 array of bit patterns."""
    import numpy as np

    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    return t.view(torch.bfloat16).to(device)


def bits_from_bf16(t: torch.Tensor):
    """numpy uint16 bit patterns of a bf16 tensor."""
    return t.detach().contiguous().cpu().view(torch.int16).numpy().view("uint16")


def release_workspace():
    """Return the current device's cached workspace (mxattn_release_workspace)."""
    _check(lib().mxattn_release_workspace(), "mxattn_release_workspace")
