"""The entry point that allocates nothing (mxattn_cross_attend_noalloc), called
through the C ABI, against mxattn_cross_attend on the same operands: the
outputs must be identical bit for bit (same kernels), on two calls in a row
with the second smaller, in every mode and on both kernel paths (streaming
keys and keys resident in LDS).  Problems beyond the static scratch are
rejected before anything is launched."""
import ctypes

import numpy as np
import pytest

from parity import log
from paper_2607_24377_amd import inputs

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def mx():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_24377_amd import mxattn

    mxattn.lib()
    return mxattn


def _operands(mx, B, H, Nq, Nkv, mode, index):
    q = inputs.generate(inputs.custom(B, H, Nq, kind="video", index=index))[0]
    _, k, v = inputs.generate(inputs.custom(B, H, Nkv, kind="video", index=index + 1))
    qt, kt, vt = (mx.bf16_from_bits(x) for x in (q, k, v))
    qc, qs = mx.quantize(qt, mx.AXIS_HEAD_DIM, mode)
    kc, ks = mx.quantize(kt, mx.AXIS_HEAD_DIM, mode)
    vc, vs = mx.quantize(vt, mx.AXIS_TOKENS, mode)
    return (qc, qs, kc, ks, vc, vs)


def _call(fn, ops, out, B, H, Nq, Nkv, mode):
    st = fn(*(t.data_ptr() for t in ops), out.data_ptr(), B, H, Nq, Nkv, 128, mode,
            torch.cuda.current_stream().cuda_stream)
    assert st == 0, st


@pytest.mark.parametrize("mode", [0, 1, 2])
def test_noalloc_equals_allocating_call_twice_second_smaller(mx, mode):
    L = mx.lib()
    # first call: 6 heads x 3000 keys (streaming kernel, 24 KiB of scratch);
    # second: 2 heads x 700 keys, then 2 heads x 300 keys (resident kernel)
    for B, H, Nq, Nkv, idx in ((1, 6, 1000, 3000, 81), (1, 2, 333, 700, 83), (2, 1, 300, 300, 85)):
        ops = _operands(mx, B, H, Nq, Nkv, mode, idx)
        want = torch.empty((B, H, Nq, 128), dtype=torch.bfloat16, device="cuda")
        got = torch.full_like(want, float("nan"))
        _call(L.mxattn_cross_attend, ops, want, B, H, Nq, Nkv, mode)
        _call(L.mxattn_cross_attend_noalloc, ops, got, B, H, Nq, Nkv, mode)
        torch.cuda.synchronize()
        log(f"[noalloc] mode {mode} B={B} H={H} Nq={Nq} Nkv={Nkv}")
        assert torch.equal(got.view(torch.int16), want.view(torch.int16)), (mode, B, H, Nq, Nkv)


def test_noalloc_at_the_720p_shape(mx):
    """40 heads x 75 600 keys (24.2 MB of scratch) on 256 queries per head."""
    B, H, Nq, Nkv, mode = 1, 40, 256, 75600, 2
    ops = _operands(mx, B, H, Nq, Nkv, mode, 87)
    want = torch.empty((B, H, Nq, 128), dtype=torch.bfloat16, device="cuda")
    got = torch.empty_like(want)
    L = mx.lib()
    _call(L.mxattn_cross_attend, ops, want, B, H, Nq, Nkv, mode)
    _call(L.mxattn_cross_attend_noalloc, ops, got, B, H, Nq, Nkv, mode)
    torch.cuda.synchronize()
    log("[noalloc] 720p shape")
    assert torch.equal(got.view(torch.int16), want.view(torch.int16))


def test_noalloc_rejects_problems_beyond_its_scratch(mx):
    L = mx.lib()
    base = 1 << 36  # never dereferenced: the size check fails first
    ops = [base + (i << 33) for i in range(7)]
    # 300 heads x ceil(14 000 / 128) = 110 tiles = 33 000 KiB > 32 MiB
    st = L.mxattn_cross_attend_noalloc(*ops, 1, 300, 1, 14000, 128, 2, None)
    assert st == 10, st
    assert b"scratch" in L.mxattn_last_error()
    # 32 768 tiles exactly fit
    assert int(np.ceil(16384 / 128)) * 256 == 32768
