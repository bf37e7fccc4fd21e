"""CPU oracle for the MXFP4 attention hot path (test infrastructure only).

Only the tests, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product library never calls it and
shares no code with it; see ``mxref.c`` for what is computed and which passage
of the paper each step follows.

Modes of the attention forward (the rows of the paper's sequential ablation
without the Hadamard rotation):

* ``ocp_vanilla``: OCP floor scale rule for Q, K, V and P~, direct placement
  (l accumulates the unquantized P~; Eq. direct_mxfp4_tile).
* ``uos``: UOS rule (Algorithm 1) everywhere, direct placement.
* ``uos_pnq``: UOS rule everywhere, Pre-Normalization Quantization
  (l accumulates the quantized P^; Eq. pnq_online_update, Algorithm 2).

``objective`` holds the data-free objective J(q) of Sec. 4.1 (E(x), D(x),
Delta(q)) used to check the boundary sweep.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "mxref.c")
_LIB_PATH = os.path.join(_HERE, "libmxref.so")

RULE_OCP, RULE_UOS, RULE_IDENTITY = 0, 1, 2
MODES = {
    "ocp_vanilla": (RULE_OCP, 0),
    "uos": (RULE_UOS, 0),
    "uos_pnq": (RULE_UOS, 1),
    "uos_pnq_rot": (RULE_UOS, 1),  # Q and K rotated by R_H before quantization
}
ROTATED = {"uos_pnq_rot"}

_lock = threading.Lock()
_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (no GPU, no HIP).  Returns the .so path."""
    if not force and os.path.exists(_LIB_PATH):
        return _LIB_PATH
    tmp = _LIB_PATH + f".tmp{os.getpid()}"
    cmd = ["gcc", "-O2", "-std=c11", "-D_GNU_SOURCE", "-fPIC", "-shared", "-pthread",
           "-ffp-contract=off", "-fno-fast-math", _SRC, "-o", tmp, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def lib() -> ctypes.CDLL:
    global _lib
    with _lock:
        if _lib is None:
            if not os.path.exists(_LIB_PATH):
                build()
            L = ctypes.CDLL(_LIB_PATH)
            P = ctypes.c_void_p
            I64 = ctypes.c_int64
            I = ctypes.c_int
            L.mxref_scale_exponent.argtypes = [ctypes.c_double, I]
            L.mxref_scale_exponent.restype = ctypes.c_long
            L.mxref_quantize_block.argtypes = [P, I, I, P, P]
            L.mxref_quantize_block.restype = I
            L.mxref_decode.argtypes = [ctypes.c_uint8, ctypes.c_uint8]
            L.mxref_decode.restype = ctypes.c_double
            L.mxref_round_bf16.argtypes = [P, I64, P]
            L.mxref_round_bf16.restype = None
            L.mxref_quantize_rows.argtypes = [P, I64, I64, I, P, P, I]
            L.mxref_quantize_rows.restype = I
            L.mxref_quantize_rows_rotated.argtypes = [P, I64, I64, I, P, P, I]
            L.mxref_quantize_rows_rotated.restype = I
            L.mxref_quantize_block_qmax.argtypes = [P, I, ctypes.c_double, P, P]
            L.mxref_quantize_block_qmax.restype = I
            L.mxref_quantize_rows_qmax.argtypes = [P, I64, I64, ctypes.c_double, P, P]
            L.mxref_quantize_rows_qmax.restype = I
            L.mxref_qmax_sse.argtypes = [P, I64, I64, I64, I, P, I, P, I]
            L.mxref_qmax_sse.restype = I
            L.mxref_softmax_rows.argtypes = [P, P, I64, I64, I64, P, I]
            L.mxref_softmax_rows.restype = I
            L.mxref_rowsum_diag.argtypes = [P, I64, I64, I64, I, ctypes.c_float, P, I]
            L.mxref_rowsum_diag.restype = I
            L.mxref_hadamard_f32.argtypes = [P, I64]
            L.mxref_hadamard_f32.restype = None
            L.mxref_quantize_keys.argtypes = [P, I64, I64, I64, I, P, P, I]
            L.mxref_quantize_keys.restype = I
            L.mxref_dequant_rows.argtypes = [P, P, I64, I64, P]
            L.mxref_dequant_rows.restype = None
            L.mxref_dequant_keys.argtypes = [P, P, I64, I64, P]
            L.mxref_dequant_keys.restype = None
            L.mxref_attention_rows.argtypes = [P, P, P, I64, I64, I64, I, I, I, I64, P, P, I]
            L.mxref_attention_rows.restype = I
            L.mxref_attention_exact_rows.argtypes = [P, P, P, I64, I64, I64, P, I]
            L.mxref_attention_exact_rows.restype = I
            L.mxref_threads.argtypes = [I]
            L.mxref_threads.restype = I
            _lib = L
    return _lib


def _ptr(a: np.ndarray) -> int:
    assert a.flags["C_CONTIGUOUS"], "oracle inputs must be C-contiguous"
    return a.ctypes.data


def threads(n: int = 0) -> int:
    """Number of host threads the oracle uses for ``nthreads=n`` (0 = all)."""
    return lib().mxref_threads(n)


# ---------------------------------------------------------------- scalars

def scale_exponent(M: float, rule: int) -> int:
    """Clamped shared-scale exponent for block maximum ``M`` (0 -> 0)."""
    return int(lib().mxref_scale_exponent(float(M), rule))


def quantize_block(values, rule: int):
    """Quantize up to 32 values.  Returns (codes uint8[n] one per element, scale byte)."""
    v = np.ascontiguousarray(np.asarray(values, dtype=np.float64))
    codes = np.zeros(v.size, dtype=np.uint8)
    sc = np.zeros(1, dtype=np.uint8)
    rc = lib().mxref_quantize_block(_ptr(v), v.size, rule, _ptr(codes), _ptr(sc))
    if rc != 0:
        raise ValueError("bad block")
    return codes, int(sc[0])


def decode(code: int, scale_byte: int) -> float:
    return float(lib().mxref_decode(code, scale_byte))


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round doubles to bf16 (nearest, ties to even); returns uint16 bits."""
    x = np.ascontiguousarray(x, dtype=np.float64)
    out = np.empty(x.shape, dtype=np.uint16)
    lib().mxref_round_bf16(_ptr(x), x.size, _ptr(out))
    return out


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


# ---------------------------------------------------------------- tensors

def quantize_rows(x_bits: np.ndarray, rule: int, nthreads: int = 0, rotate: bool = False):
    """Blocks along the last axis.  x_bits: bf16 bits [..., d].  With rotate,
    each row is first multiplied by R_H (hadamard_f32, d = 128 only).

    Returns codes [..., d/2] and scales [..., d/32] (uint8)."""
    x = np.ascontiguousarray(x_bits, dtype=np.uint16)
    d = x.shape[-1]
    rows = x.size // d
    codes = np.empty(x.shape[:-1] + (d // 2,), dtype=np.uint8)
    scales = np.empty(x.shape[:-1] + (d // 32,), dtype=np.uint8)
    fn = lib().mxref_quantize_rows_rotated if rotate else lib().mxref_quantize_rows
    rc = fn(_ptr(x), rows, d, rule, _ptr(codes), _ptr(scales), nthreads)
    if rc != 0:
        raise ValueError("oracle row quantizer rejected its arguments")
    return codes, scales


def quantize_block_qmax(values, q: float):
    """Quantize up to 32 values with the ceil rule of boundary q (4 <= q <= 8)."""
    v = np.ascontiguousarray(np.asarray(values, dtype=np.float64))
    codes = np.zeros(v.size, dtype=np.uint8)
    sc = np.zeros(1, dtype=np.uint8)
    if lib().mxref_quantize_block_qmax(_ptr(v), v.size, float(q), _ptr(codes), _ptr(sc)) != 0:
        raise ValueError("bad block or boundary")
    return codes, int(sc[0])


def quantize_rows_qmax(x_bits: np.ndarray, q: float):
    """Blocks along the last axis with the ceil rule of boundary q."""
    x = np.ascontiguousarray(x_bits, dtype=np.uint16)
    d = x.shape[-1]
    rows = x.size // d
    codes = np.empty(x.shape[:-1] + (d // 2,), dtype=np.uint8)
    scales = np.empty(x.shape[:-1] + (d // 32,), dtype=np.uint8)
    if lib().mxref_quantize_rows_qmax(_ptr(x), rows, d, float(q), _ptr(codes), _ptr(scales)) != 0:
        raise ValueError("bad arguments")
    return codes, scales


def qmax_sse(x_bits: np.ndarray, axis: int, qs, nthreads: int = 0) -> np.ndarray:
    """Per-head sum of squared MXFP4 errors for each boundary in qs.

    x_bits: bf16 bits [..., N, d]; axis 3 = blocks along d, 2 = along tokens.
    Returns [heads, len(qs)] fp64."""
    x = np.ascontiguousarray(x_bits, dtype=np.uint16)
    N, d = x.shape[-2], x.shape[-1]
    heads = x.size // (N * d)
    q = np.ascontiguousarray(np.asarray(qs, dtype=np.float64))
    out = np.empty((heads, q.size), dtype=np.float64)
    if lib().mxref_qmax_sse(_ptr(x), heads, N, d, axis, _ptr(q), q.size, _ptr(out), nthreads) != 0:
        raise ValueError("bad arguments")
    return out


DIAG_FIELDS = ("rowsum", "mass", "zeroing", "saturation", "down", "up", "exact", "entropy")


def softmax_rows(q: np.ndarray, k: np.ndarray, nthreads: int = 0) -> np.ndarray:
    """Exact fp64 softmax(q k^T / sqrt(d)) rows; q [rows, d], k [N, d] (float)."""
    qd = np.ascontiguousarray(q, dtype=np.float64)
    kd = np.ascontiguousarray(k, dtype=np.float64)
    out = np.empty((qd.shape[0], kd.shape[0]), dtype=np.float64)
    if lib().mxref_softmax_rows(_ptr(qd), _ptr(kd), kd.shape[0], kd.shape[1], qd.shape[0], _ptr(out),
                                nthreads) != 0:
        raise ValueError("bad arguments")
    return out


def rowsum_diag(P: np.ndarray, N: int, rule: int, gamma: float = 1.0, nthreads: int = 0) -> np.ndarray:
    """Per-row diagnostics of MXFP4-quantizing fp32 probability rows P [rows, ld]
    (first N entries valid); returns [rows, 8] fp64 in DIAG_FIELDS order."""
    p = np.ascontiguousarray(P, dtype=np.float32)
    rows, ld = p.shape
    out = np.empty((rows, 8), dtype=np.float64)
    if lib().mxref_rowsum_diag(_ptr(p), rows, N, ld, rule, float(gamma), _ptr(out), nthreads) != 0:
        raise ValueError("bad arguments")
    return out


def hadamard_f32(x: np.ndarray) -> np.ndarray:
    """x R_H row by row (fp32 in, fp32 out), the oracle's fixed rotation."""
    y = np.array(x, dtype=np.float32, order="C", copy=True)
    d = y.shape[-1]
    for row in y.reshape(-1, d):
        lib().mxref_hadamard_f32(_ptr(row), d)
    return y


def quantize_keys(x_bits: np.ndarray, rule: int, nthreads: int = 0):
    """Blocks along the token axis.  x_bits: bf16 bits [..., N, d].

    Returns codes [..., d, nb*16] and scales [..., d, nb], nb = ceil(N/32)."""
    x = np.ascontiguousarray(x_bits, dtype=np.uint16)
    N, d = x.shape[-2], x.shape[-1]
    heads = x.size // (N * d)
    nb = (N + 31) // 32
    codes = np.empty(x.shape[:-2] + (d, nb * 16), dtype=np.uint8)
    scales = np.empty(x.shape[:-2] + (d, nb), dtype=np.uint8)
    rc = lib().mxref_quantize_keys(_ptr(x), heads, N, d, rule, _ptr(codes), _ptr(scales), nthreads)
    if rc != 0:
        raise ValueError("mxref_quantize_keys rejected its arguments")
    return codes, scales


def dequant_rows(codes: np.ndarray, scales: np.ndarray) -> np.ndarray:
    codes = np.ascontiguousarray(codes, dtype=np.uint8)
    scales = np.ascontiguousarray(scales, dtype=np.uint8)
    d = codes.shape[-1] * 2
    rows = codes.size // (d // 2)
    out = np.empty(codes.shape[:-1] + (d,), dtype=np.float64)
    lib().mxref_dequant_rows(_ptr(codes), _ptr(scales), rows, d, _ptr(out))
    return out


def dequant_keys(codes: np.ndarray, scales: np.ndarray, N: int) -> np.ndarray:
    """One head: codes [d, nb*16], scales [d, nb] -> [N, d] doubles."""
    codes = np.ascontiguousarray(codes, dtype=np.uint8)
    scales = np.ascontiguousarray(scales, dtype=np.uint8)
    d = codes.shape[0]
    out = np.empty((N, d), dtype=np.float64)
    lib().mxref_dequant_keys(_ptr(codes), _ptr(scales), N, d, _ptr(out))
    return out


def attention_rows(q: np.ndarray, k: np.ndarray, v: np.ndarray, p_rule: int, pnq: int,
                   exact: int = 0, block_c: int = 128, diag: bool = False, nthreads: int = 0):
    """Tiled online-softmax attention of the given query rows against one head.

    q [R, d], k [N, d], v [N, d] (doubles).  Returns O [R, d] in fp64 and, if
    ``diag``, a [R, 8] array (l, induced row sum, unrolled l, max |O - O_unrolled|,
    tiles, max rises, P~ elements within 4 fp32 ulps of an E2M1 decision
    threshold, blocks whose maximum is within 4 fp32 ulps of an end of the
    scale rule's range)."""
    q = np.ascontiguousarray(q, dtype=np.float64)
    k = np.ascontiguousarray(k, dtype=np.float64)
    v = np.ascontiguousarray(v, dtype=np.float64)
    R, d = q.shape
    N = k.shape[0]
    assert k.shape == (N, d) and v.shape == (N, d)
    out = np.empty((R, d), dtype=np.float64)
    dg = np.empty((R, 8), dtype=np.float64) if diag else None
    rc = lib().mxref_attention_rows(_ptr(q), _ptr(k), _ptr(v), N, d, R, p_rule, pnq, exact,
                                    block_c, _ptr(out), _ptr(dg) if diag else None, nthreads)
    if rc != 0:
        raise ValueError("mxref_attention_rows rejected its arguments")
    return (out, dg) if diag else out


def attention_exact_rows(q: np.ndarray, k: np.ndarray, v: np.ndarray, nthreads: int = 0):
    """softmax(q k^T / sqrt(d)) v in fp64 (Eq. standard_attention)."""
    q = np.ascontiguousarray(q, dtype=np.float64)
    k = np.ascontiguousarray(k, dtype=np.float64)
    v = np.ascontiguousarray(v, dtype=np.float64)
    R, d = q.shape
    N = k.shape[0]
    out = np.empty((R, d), dtype=np.float64)
    rc = lib().mxref_attention_exact_rows(_ptr(q), _ptr(k), _ptr(v), N, d, R, _ptr(out), nthreads)
    if rc != 0:
        raise ValueError("mxref_attention_exact_rows rejected its arguments")
    return out


# ---------------------------------------------------------------- high level

def quantize_qkv(q_bits, k_bits, v_bits, mode: str, nthreads: int = 0):
    """Quantize bf16 Q/K (blocks along d) and V (blocks along tokens) for a mode.

    Inputs are bf16 bits [B, H, N, d].  Returns a dict of codes/scales in the
    library's public layouts."""
    rule = MODES[mode][0]
    rot = mode in ROTATED
    qc, qs = quantize_rows(q_bits, rule, nthreads, rotate=rot)
    kc, ks = quantize_rows(k_bits, rule, nthreads, rotate=rot)
    vc, vs = quantize_keys(v_bits, rule, nthreads)
    return dict(qc=qc, qs=qs, kc=kc, ks=ks, vc=vc, vs=vs)


def mx_attention_head_rows(qc, qs, kc, ks, vc, vs, N: int, rows, mode: str, block_c: int = 128,
                           diag: bool = False, nthreads: int = 0):
    """MXFP4 attention for query ``rows`` of ONE head from its codes/scales.

    qc/kc [N, d/2], qs/ks [N, d/32], vc [d, nb*16], vs [d, nb].  Returns fp64
    O rows (and diagnostics if asked)."""
    p_rule, pnq = MODES[mode]
    rows = np.asarray(rows, dtype=np.int64)
    qh = dequant_rows(np.ascontiguousarray(qc[rows]), np.ascontiguousarray(qs[rows]))
    kh = dequant_rows(kc, ks)
    vh = dequant_keys(vc, vs, N)
    return attention_rows(qh, kh, vh, p_rule, pnq, 0, block_c, diag, nthreads)
