"""The C-ABI library loads, exports every entry point its header declares, and
rejects bad arguments before touching the GPU (these run without one)."""
import ctypes
import os
import re

import pytest

from conftest import ROOT

HEADER = os.path.join(ROOT, "include", "mxattn.h")


def _declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mxattn_\w+)\s*\(", text)))


@pytest.fixture(scope="module")
def L():
    from paper_2607_24377_amd import mxattn

    if not os.path.exists(mxattn.LIB_PATH):
        from paper_2607_24377_amd import build

        build.build()
    return mxattn.lib()


def test_header_declares_the_entry_points():
    names = _declared_functions()
    for n in ["mxattn_quantize", "mxattn_forward", "mxattn_attend", "mxattn_codes_bytes",
              "mxattn_quantize_qmax", "mxattn_qmax_sse",
              "mxattn_scales_bytes", "mxattn_kv_tile", "mxattn_status_string",
              "mxattn_last_error", "mxattn_release_workspace"]:
        assert n in names


def test_library_exports_every_declared_symbol(L):
    for name in _declared_functions():
        assert hasattr(L, name), name
        getattr(L, name)  # resolves


def test_queries(L):
    assert L.mxattn_version() >= 100
    assert L.mxattn_kv_tile() in (32, 64, 128, 256)  # whole 32-key MXFP4 blocks
    assert L.mxattn_query_tile() > 0
    B, H, N, d = 1, 40, 75600, 128
    assert L.mxattn_codes_bytes(3, B, H, N, d) == B * H * N * 64
    assert L.mxattn_scales_bytes(3, B, H, N, d) == B * H * N * 4
    nb = (N + 31) // 32
    assert L.mxattn_codes_bytes(2, B, H, N, d) == B * H * d * nb * 16
    assert L.mxattn_scales_bytes(2, B, H, N, d) == B * H * d * nb
    assert L.mxattn_codes_bytes(1, B, H, N, d) == 0
    assert L.mxattn_codes_bytes(3, B, H, N, 64) == 0
    for s in range(0, 9):
        assert L.mxattn_status_string(s)
    assert L.mxattn_status_string(0) == b"ok"


FAKE = 0x100000  # a 16-byte aligned non-null address; never dereferenced


def test_quantize_rejects_bad_arguments(L):
    q = L.mxattn_quantize
    assert q(None, FAKE, FAKE, 3, 2, 1, 1, 8, 128, None) == 1          # NULL
    assert q(FAKE, FAKE, None, 3, 2, 1, 1, 8, 128, None) == 1
    assert q(FAKE, FAKE, FAKE, 1, 2, 1, 1, 8, 128, None) == 5          # AXIS
    assert q(FAKE, FAKE, FAKE, 3, 4, 1, 1, 8, 128, None) == 4          # MODE
    assert q(FAKE, FAKE, FAKE, 3, 3, 0, 1, 8, 128, None) == 2          # mode 3 (rotated) is valid
    assert q(FAKE, FAKE, FAKE, 3, -1, 1, 1, 8, 128, None) == 4
    assert q(FAKE, FAKE, FAKE, 3, 2, 0, 1, 8, 128, None) == 2          # SHAPE
    assert q(FAKE, FAKE, FAKE, 2, 2, 1, 1, 0, 128, None) == 2
    assert q(FAKE, FAKE, FAKE, 3, 2, 1, 1, 1 << 29, 128, None) == 2
    assert q(FAKE, FAKE, FAKE, 3, 2, 1, 1, 8, 64, None) == 6           # UNSUPPORTED
    assert q(FAKE + 2, FAKE, FAKE, 3, 2, 1, 1, 8, 128, None) == 3      # ALIGN
    assert q(FAKE, FAKE + 8, FAKE, 3, 2, 1, 1, 8, 128, None) == 3


def test_element_count_limit(L):
    """At most 2^35 elements per tensor (every grid stays below 2^31
    workgroups); the byte-size queries return 0 beyond it."""
    q = L.mxattn_quantize
    assert q(FAKE, FAKE, FAKE, 3, 2, 1 << 8, 1 << 8, 1 << 20, 128, None) == 2
    assert L.mxattn_codes_bytes(3, 1 << 8, 1 << 8, 1 << 20, 128) == 0
    assert L.mxattn_codes_bytes(3, 1 << 8, 1 << 8, 1 << 12, 128) == (1 << 28) * 64


def test_forward_and_attend_reject_bad_arguments(L):
    f = L.mxattn_forward
    assert f(None, FAKE, FAKE, FAKE, 1, 1, 8, 128, 2, None) == 1
    assert f(FAKE, FAKE, FAKE, None, 1, 1, 8, 128, 2, None) == 1
    assert f(FAKE, FAKE, FAKE, FAKE, 1, 1, 8, 128, 7, None) == 4
    assert f(FAKE, FAKE, FAKE, FAKE, 1, 0, 8, 128, 2, None) == 2
    assert f(FAKE, FAKE, FAKE, FAKE, 1, 1, -5, 128, 2, None) == 2
    assert f(FAKE, FAKE, FAKE, FAKE, 1, 1, 8, 256, 2, None) == 6
    assert f(FAKE, FAKE, FAKE + 4, FAKE, 1, 1, 8, 128, 2, None) == 3
    c = L.mxattn_cross_forward
    assert c(FAKE, FAKE, FAKE, FAKE, 1, 1, 8, 0, 128, 2, None) == 2    # Nkv < 1
    assert c(FAKE, FAKE, FAKE, FAKE, 1, 1, 0, 8, 128, 2, None) == 2    # Nq < 1
    assert c(FAKE, None, FAKE, FAKE, 1, 1, 8, 8, 128, 2, None) == 1
    assert c(FAKE, FAKE, FAKE, FAKE, 1, 1, 8, 8, 128, 5, None) == 4
    # the fused kernel's key limit (2^24) and query-tile count (2^30), checked
    # before any allocation or launch (the quantizer alone accepts N up to 2^28)
    assert c(FAKE, FAKE, FAKE, FAKE, 1, 1, 8, (1 << 24) + 1, 128, 2, None) == 2
    assert f(FAKE, FAKE, FAKE, FAKE, 1, 1, (1 << 24) + 1, 128, 2, None) == 2
    assert c(FAKE, FAKE, FAKE, FAKE, 1 << 10, 1 << 10, (1 << 17) + 1, 8, 128, 2, None) == 2
    ca = L.mxattn_cross_attend
    assert ca(*([FAKE] * 7), 1, 1, 8, 1 << 29, 128, 2, None) == 2
    assert ca(*([FAKE] * 7), 1, 1, 8, (1 << 24) + 1, 128, 2, None) == 2
    assert ca(*([FAKE] * 7), 1, 1, 8, 8, 64, 2, None) == 6
    a = L.mxattn_attend
    args = [FAKE] * 7
    bad = list(args)
    bad[3] = None
    assert a(*bad, 1, 1, 8, 128, 0, None) == 1
    assert a(*args, 1, 1, 8, 128, 9, None) == 4
    assert a(*args, 1, 1, 0, 128, 0, None) == 2
    bad = list(args)
    bad[3] = FAKE + 2  # k_scales must be 4-byte aligned
    assert a(*bad, 1, 1, 8, 128, 0, None) == 3
    bad = list(args)
    bad[1] = FAKE + 1  # q_scales may have any alignment: only the shape error fires
    assert a(*bad, 1, 1, 0, 128, 0, None) == 2


def test_output_overlapping_an_input_is_rejected(L):
    """`out` sharing a byte with an input is a shape error, caught before any
    allocation or launch.  Only overlapping cases are called: the pointers
    are not device memory."""
    B, H, N, d = 1, 2, 64, 128
    nb = B * H * N * d * 2  # bf16 bytes of one [B, H, N, d] tensor
    q, k, v = FAKE, FAKE + (1 << 24), FAKE + (2 << 24)
    f, c = L.mxattn_forward, L.mxattn_cross_forward
    assert f(q, k, v, q, B, H, N, d, 2, None) == 2
    assert f(q, k, v, q + nb - 16, B, H, N, d, 2, None) == 2   # last 16 bytes of q
    assert f(q, k, v, k - nb + 16, B, H, N, d, 2, None) == 2   # first 16 bytes of k
    assert f(q, k, v, v + 1024, B, H, N, d, 0, None) == 2
    # cross-attention: out [B, H, Nq, d] against k, v [B, H, Nkv, d]
    Nq, Nkv = 256, 16
    assert c(q, k, v, k - B * H * Nq * d * 2 + 16, B, H, Nq, Nkv, d, 2, None) == 2
    assert c(q, k, v, v + B * H * Nkv * d * 2 - 16, B, H, Nq, Nkv, d, 1, None) == 2
    # quantized operands: codes and scales of Q, K and V
    a, ca = L.mxattn_attend, L.mxattn_cross_attend
    ops = [FAKE + (i << 24) for i in range(6)]  # qc, qs, kc, ks, vc, vs
    for i in range(6):
        assert a(*ops, ops[i], B, H, N, d, 2, None) == 2, i
    qs_bytes = B * H * Nq * 4
    assert ca(*ops, ops[1] - B * H * Nq * d * 2 + 16, B, H, Nq, Nkv, d, 2, None) == 2
    assert ca(*ops, ops[1] + qs_bytes - 16, B, H, Nq, Nkv, d, 2, None) == 2


def test_boundary_entry_points_reject_bad_arguments(L):
    q = L.mxattn_quantize_qmax
    assert q(FAKE, FAKE, FAKE, 3, 7.25, 1, 1, 0, 128, None) == 2       # shape: valid q
    assert q(None, FAKE, FAKE, 3, 7.25, 1, 1, 8, 128, None) == 1
    assert q(FAKE, FAKE, FAKE, 1, 7.25, 1, 1, 8, 128, None) == 5
    for bad in (3.999, 8.001, float("nan"), float("inf"), -7.25):
        assert q(FAKE, FAKE, FAKE, 3, bad, 1, 1, 8, 128, None) == 9    # BOUNDARY
    assert q(FAKE, FAKE, FAKE, 2, 4.0, 1, 1, 8, 64, None) == 6         # q = 4 and 8 are valid
    assert q(FAKE, FAKE + 4, FAKE, 3, 8.0, 1, 1, 8, 128, None) == 3
    s = L.mxattn_qmax_sse
    qs = (ctypes.c_double * 65)(*([7.0] * 65))
    assert s(FAKE, 3, qs, 41, FAKE, 1, 1, 0, 128, None) == 2
    assert s(FAKE, 3, None, 1, FAKE, 1, 1, 8, 128, None) == 1
    assert s(FAKE, 3, qs, 1, None, 1, 1, 8, 128, None) == 1
    assert s(FAKE, 4, qs, 1, FAKE, 1, 1, 8, 128, None) == 5
    assert s(FAKE, 3, qs, 0, FAKE, 1, 1, 8, 128, None) == 9
    assert s(FAKE, 3, qs, 65, FAKE, 1, 1, 8, 128, None) == 9
    bad = (ctypes.c_double * 3)(6.0, 8.5, 7.0)
    assert s(FAKE, 2, bad, 3, FAKE, 1, 1, 8, 128, None) == 9
    assert s(FAKE, 3, qs, 64, FAKE + 4, 1, 1, 8, 128, None) == 3       # sse needs 8 bytes
    assert s(FAKE, 3, qs, 64, FAKE, 1, 1, 8, 96, None) == 6


def test_rowsum_entry_points_reject_bad_arguments(L):
    s = L.mxattn_softmax_rows
    assert s(None, FAKE, FAKE, 1, 1, 8, 8, 128, 0, 8, 8, None) == 1
    assert s(FAKE, FAKE, FAKE, 1, 1, 8, 8, 128, 4, 5, 8, None) == 2     # rows past Nq
    assert s(FAKE, FAKE, FAKE, 1, 1, 8, 8, 128, 0, 0, 8, None) == 2     # no rows
    assert s(FAKE, FAKE, FAKE, 1, 1, 8, 8, 128, 0, 8, 6, None) == 2     # ld < Nkv
    assert s(FAKE, FAKE, FAKE, 1, 1, 8, 10, 128, 0, 8, 10, None) == 2   # ld % 4
    assert s(FAKE, FAKE, FAKE, 1, 1, 8, 8, 64, 0, 8, 8, None) == 6
    assert s(FAKE, FAKE, FAKE + 4, 1, 1, 8, 8, 128, 0, 8, 8, None) == 3
    d = L.mxattn_rowsum_diag
    assert d(None, 4, 8, 8, 1, 1.0, FAKE, None) == 1
    assert d(FAKE, 4, 8, 8, 9, 1.0, FAKE, None) == 4
    assert d(FAKE, 0, 8, 8, 1, 1.0, FAKE, None) == 2
    assert d(FAKE, 4, 9, 8, 1, 1.0, FAKE, None) == 2                     # ld < N
    assert d(FAKE, 4, 8, 8, 1, 0.0, FAKE, None) == 9                     # gamma
    assert d(FAKE, 4, 8, 8, 1, float("nan"), FAKE, None) == 9
    assert d(FAKE + 8, 4, 8, 8, 1, 1.0, FAKE, None) == 3
    assert d(FAKE, 4, 8, 8, 1, 1.0, FAKE + 4, None) == 3
    a = L.mxattn_attention_rowsum_diag
    assert a(FAKE, FAKE, 1, 1, 8, 8, 128, 1, 1.0, None, None) == 1
    assert a(FAKE, FAKE, 1, 1, 0, 8, 128, 1, 1.0, FAKE, None) == 2
    assert a(FAKE, FAKE, 1, 1, 8, 8, 128, 7, 1.0, FAKE, None) == 4
    assert a(FAKE, FAKE, 1, 1, 8, 8, 128, 1, -1.0, FAKE, None) == 9
