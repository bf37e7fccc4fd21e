"""Generic scale boundary q on the GPU against the oracle.

* mxattn_quantize_qmax: codes and scales bit-exact, both block axes, for the
  named boundaries (TFS 6, OAS 7, UOS 7.25, the ceil form of OCP 8, the
  family's end 4) and points of the 6.00-8.00 sweep: every finite bf16 value
  as a block maximum and as an element, random rows spanning the exponent
  range, a ragged token axis, and the workloads' Q, K, V.
* mxattn_qmax_sse: per-head sums of squared errors against the oracle's sweep
  on small ragged tensors (all 41 boundaries) and on sampled heads of the
  720p workload, with |gpu - oracle| <= 1e-6 * oracle + 1e-24 * sum(x^2).
  The oracle sums in fp64; the GPU sums groups of 8 exact squared errors in
  fp32 (exact unless an element rounds to zero with low-order bits, else off
  by at most 7 * 2^-24 = 4.2e-7 of the group) and the groups in fp64.  The
  second term admits elements far below their block's scale, whose scaled
  value x 2^-e the GPU forms in fp32.
* The sweep's per-head optimum over the 41 boundaries for Q, K and V of every
  workload (the analogue of Table cx_distribution on the synthetic inputs),
  logged.
"""
import collections

import numpy as np
import pytest

import oracle
from parity import log, workload_bits
from paper_2607_24377_amd import inputs

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

SWEEP = [round(6.0 + 0.05 * i, 2) for i in range(41)]
NAMED = [4.0, 6.0, 7.0, 7.25, 8.0]
REL_TOL, ENERGY_TOL = 1e-6, 1e-24


@pytest.fixture(scope="module")
def mx():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_24377_amd import mxattn

    mxattn.lib()
    return mxattn


def _finite_bf16():
    b = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    return b[((b >> 7) & 0xFF) != 0xFF]


def _token_rows(x_bits):
    """Token blocks of x [B, H, N, d] as rows: [B*H, d, N padded to 32]
    (the library's token layout is the head-dim layout of this transpose)."""
    B, H, N, d = x_bits.shape
    pad = (-N) % 32
    xt = np.swapaxes(x_bits.reshape(B * H, N, d), 1, 2)
    return np.concatenate([xt, np.zeros((B * H, d, pad), np.uint16)], axis=2)


def _check_quant(mx, x_bits, axis, q, label):
    codes, scales = mx.quantize_qmax(mx.bf16_from_bits(x_bits), axis, q)
    if axis == mx.AXIS_HEAD_DIM:
        oc, os_ = oracle.quantize_rows_qmax(x_bits, q)
    else:
        oc, os_ = oracle.quantize_rows_qmax(_token_rows(x_bits), q)
        oc, os_ = oc.reshape(codes.shape), os_.reshape(scales.shape)
    gs, gc = scales.cpu().numpy(), codes.cpu().numpy()
    assert np.array_equal(gs, os_), f"{label} q={q}: scales differ at {np.argwhere(gs != os_)[:5]}"
    assert np.array_equal(gc, oc), f"{label} q={q}: codes differ at {np.argwhere(gc != oc)[:5]}"


@pytest.mark.parametrize("q", NAMED + [6.05, 6.5, 7.2, 7.3, 7.95])
def test_quantize_every_bf16_as_maximum_and_element(mx, q):
    log(f"[qmax quant exhaustive] q={q}")
    bits = _finite_bf16()
    n = bits.size
    x = np.zeros((n, 32), np.uint16)
    x[:, 0] = bits                      # every value as a block maximum candidate
    x[:, 9] = bits[::-1]
    x[:, 20] = np.roll(bits, 12345)     # and as a small element of another block
    pad = (-n) % 4
    xx = np.concatenate([x, np.zeros((pad, 32), np.uint16)]).reshape(1, 1, -1, 128)
    _check_quant(mx, xx, mx.AXIS_HEAD_DIM, q, "exhaustive head-dim")
    # the same tensor with blocks along the tokens, whole and with a ragged end
    _check_quant(mx, xx, mx.AXIS_TOKENS, q, "exhaustive tokens")
    _check_quant(mx, np.ascontiguousarray(xx[:, :, :16300]), mx.AXIS_TOKENS, q, "exhaustive tokens ragged")


@pytest.mark.parametrize("q", NAMED + SWEEP[1::4])
def test_quantize_random_rows_and_ragged_tokens(mx, q):
    rng = np.random.default_rng(int(q * 100))
    rows = 4096
    mag = np.exp2(rng.integers(-130, 120, size=(rows, 1))).astype(np.float32)
    x = rng.standard_t(3, (rows, 128)).astype(np.float32) * mag
    x[::53] = 0.0
    x[1::71, 5:] = 0.0
    bits = inputs.f32_to_bf16_bits(x)
    log(f"[qmax quant random] q={q}")
    _check_quant(mx, bits.reshape(2, 2, rows // 4, 128), mx.AXIS_HEAD_DIM, q, "random rows")
    for N in (77, 1000):
        xr = bits[: 2 * N].reshape(1, 2, N, 128)
        _check_quant(mx, xr, mx.AXIS_TOKENS, q, f"tokens N={N}")


def test_uos_boundary_matches_uos_quantizer(mx):
    q_, k_, v_ = workload_bits(1)
    for axis, x in ((mx.AXIS_HEAD_DIM, k_), (mx.AXIS_TOKENS, v_)):
        t = mx.bf16_from_bits(x)
        a = mx.quantize_qmax(t, axis, 7.25)
        b = mx.quantize(t, axis, "uos")
        assert torch.equal(a[0], b[0]) and torch.equal(a[1], b[1])


@pytest.mark.parametrize("cfg", [0, 4])
@pytest.mark.parametrize("q", [6.0, 7.0, 8.0])
def test_quantize_workload_tensors(mx, cfg, q):
    qb, kb, vb = workload_bits(cfg)
    w = inputs.workload(cfg)
    log(f"[qmax quant workload] {w.name} q={q}")
    _check_quant(mx, qb, mx.AXIS_HEAD_DIM, q, f"{w.name} q")
    _check_quant(mx, kb, mx.AXIS_HEAD_DIM, q, f"{w.name} k")
    _check_quant(mx, vb, mx.AXIS_TOKENS, q, f"{w.name} v")


def _check_sse(got, ref, x_bits, label):
    heads = ref.shape[0]
    energy = (oracle.bf16_to_f64(x_bits).reshape(heads, -1) ** 2).sum(axis=1)
    err = np.abs(got - ref)
    bound = REL_TOL * ref + ENERGY_TOL * energy[:, None]
    worst = float(np.max(err / np.maximum(bound, 1e-300)))
    log(f"[qmax sse] {label}: worst error / bound {worst:.3g}")
    assert np.all(np.isfinite(got)) and np.all(err <= bound), label


@pytest.mark.parametrize("axis", [2, 3])
@pytest.mark.parametrize("N", [1, 31, 200, 1027])
def test_sse_small_ragged_all_boundaries(mx, axis, N):
    rng = np.random.default_rng(N * 7 + axis)
    mag = np.exp2(rng.integers(-40, 40, size=(3, 1, 1))).astype(np.float32)
    x = rng.standard_t(4, (3, N, 128)).astype(np.float32) * mag
    x[1, ::5] = 0.0
    if N > 8:
        x[2, 3] *= 2.0 ** 60  # a row far above the rest of its head
    bits = inputs.f32_to_bf16_bits(x).reshape(1, 3, N, 128)
    qs = SWEEP + NAMED
    got = mx.qmax_sse(mx.bf16_from_bits(bits), axis, qs).cpu().numpy()
    ref = oracle.qmax_sse(bits, axis, qs)
    _check_sse(got, ref, bits, f"axis {axis} N={N}")


def test_sse_wide_exponent_range(mx):
    rng = np.random.default_rng(31)
    rows = 2048
    mag = np.exp2(rng.integers(-128, 100, size=(rows, 1))).astype(np.float32)
    x = rng.standard_t(3, (rows, 128)).astype(np.float32) * mag
    bits = inputs.f32_to_bf16_bits(x).reshape(1, 4, rows // 4, 128)
    for axis in (2, 3):
        got = mx.qmax_sse(mx.bf16_from_bits(bits), axis, NAMED).cpu().numpy()
        ref = oracle.qmax_sse(bits, axis, NAMED)
        _check_sse(got, ref, bits, f"wide range axis {axis}")


def test_sse_argument_checks(mx):
    x = mx.bf16_from_bits(np.zeros((1, 1, 32, 128), np.uint16))
    for bad in ([3.99], [8.01], [float("nan")], [], [7.0] * 65):
        with pytest.raises(mx.MxattnError):
            mx.qmax_sse(x, 3, bad)
    with pytest.raises(mx.MxattnError):
        mx.quantize_qmax(x, 3, 8.5)
    with pytest.raises(mx.MxattnError):
        mx.qmax_sse(x, 1, [7.25])


def test_sse_720p_sampled_heads(mx):
    qb, kb, vb = workload_bits(3)
    w = inputs.workload(3)
    qs = [6.0, 6.5, 7.0, 7.2, 7.25, 7.3, 8.0]
    heads = [0, 17, 39]
    for name, x, axis in (("q", qb, 3), ("k", kb, 3), ("v", vb, 2)):
        log(f"[qmax sse 720p] {name}")
        got = mx.qmax_sse(mx.bf16_from_bits(x), axis, qs).cpu().numpy()
        sub = np.ascontiguousarray(x[:, heads])
        ref = oracle.qmax_sse(sub, axis, qs)
        _check_sse(got[heads], ref, sub, f"{w.name} {name}")
        torch.cuda.empty_cache()


def test_workload_optimum_distribution(mx):
    """Per-head optimum of the sweep for Q, K, V of every workload (logged)."""
    table = {}
    for cfg in range(5):
        w = inputs.workload(cfg)
        qb, kb, vb = workload_bits(cfg)
        for name, x, axis in (("Q", qb, 3), ("K", kb, 3), ("V", vb, 2)):
            sse = mx.qmax_sse(mx.bf16_from_bits(x), axis, SWEEP).cpu().numpy()
            best = [SWEEP[i] for i in np.argmin(sse, axis=1)]
            table[(w.name, name)] = collections.Counter(best)
            assert all(6.0 <= b <= 8.0 for b in best)
        torch.cuda.empty_cache()
    for (wname, t), cnt in table.items():
        tot = sum(cnt.values())
        top = ", ".join(f"{q:.2f}: {100.0 * c / tot:.1f}%" for q, c in cnt.most_common(4))
        log(f"[qmax optimum] {wname} {t} ({tot} heads): {top}")
