"""Row-sum diagnostics on the GPU against the oracle (Sec. 5.5, "Validation
of Pre-Normalization Quantization", Fig. pnq_rowsum).

* mxattn_softmax_rows against the oracle's fp64 softmax of the same bf16 Q, K:
  relative error of every entry within a bound derived from the arithmetic
  (fp32 accumulation of 128 exact bf16 products on the matrix cores, the
  fp32 normalizer over the lane's keys, the exponential's rounding), entries
  below 2^-120 excepted (the GPU flushes below 2^-126).
* mxattn_rowsum_diag against the oracle on the same fp32 rows: every entry is
  classified and rounded identically, so the fp64 sums differ only in the
  order of additions (|diff| <= 1e-11 on these row masses); the entropy uses
  the fp32 base-2 logarithm (relative 1e-6).  Random peaked and flat rows,
  ragged N with junk past N, uniform, one-hot and zero rows, both scale
  rules, pre-scales 1, 2 and 1.37.
* mxattn_attention_rowsum_diag (probabilities quantized in registers, never
  materialized) equals the two calls composed up to the order of the fp64
  additions (1e-11), at 720p as well as small and ragged sizes.
* A summary of the statistics the paper reports, for the synthetic workloads
  (logged).
"""
import math

import numpy as np
import pytest

import oracle
from parity import log, workload_bits
from paper_2607_24377_amd import inputs

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

U = 2.0 ** -24
C = 0.12751743082459868  # log2(e) / sqrt(128)
MODES = {"uos": oracle.RULE_UOS, "ocp_vanilla": oracle.RULE_OCP}


@pytest.fixture(scope="module")
def mx():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_24377_amd import mxattn

    mxattn.lib()
    return mxattn


def _softmax_check(mx, q_bits, k_bits, row0, rows, label):
    """q_bits [1, H, Nq, 128], k_bits [1, H, Nkv, 128]."""
    H, Nkv = q_bits.shape[1], k_bits.shape[2]
    P = mx.softmax_rows(mx.bf16_from_bits(q_bits), mx.bf16_from_bits(k_bits), row0, rows).cpu().numpy()
    worst = 0.0
    for h in range(H):
        q = oracle.bf16_to_f64(q_bits[0, h, row0:row0 + rows])
        k = oracle.bf16_to_f64(k_bits[0, h])
        ref = oracle.softmax_rows(q, k)
        got = P[0, h, :, :Nkv].astype(np.float64)
        A = np.abs(q) @ np.abs(k).T                       # sum_k |q_k k_k| per score
        bound = (math.log(2) * C * 127 * U * (A + A.max(axis=1, keepdims=True))
                 + (Nkv / 32 + 48) * U + 4 * U)
        big = ref > 2.0 ** -120
        rel = np.abs(got[big] / ref[big] - 1.0)
        assert np.all(rel <= bound[big]), f"{label} head {h}: worst {np.max(rel / bound[big]):.3g} of bound"
        assert np.all(got[~big] <= 2.0 ** -119), label
        worst = max(worst, float(np.max(rel / bound[big])))
    log(f"[softmax rows] {label}: worst relative error / bound {worst:.3g}")


@pytest.mark.parametrize("cfg", [0])
def test_softmax_rows_tiny(mx, cfg):
    q, k, _ = workload_bits(cfg)
    _softmax_check(mx, q, k, 0, q.shape[2], "tiny all rows")
    _softmax_check(mx, q, k, 100, 37, "tiny rows 100..136")


@pytest.mark.parametrize("nq,nkv", [(1, 1), (5, 31), (130, 333), (257, 1000)])
def test_softmax_rows_ragged(mx, nq, nkv):
    w = inputs.custom(1, 2, max(nq, nkv), kind="video", index=31)
    q, k, _ = inputs.generate(w)
    _softmax_check(mx, np.ascontiguousarray(q[:, :, :nq]), np.ascontiguousarray(k[:, :, :nkv]), 0, nq,
                   f"Nq={nq} Nkv={nkv}")


def test_softmax_rows_720p_slice(mx):
    q, k, _ = workload_bits(3)
    sub_q = np.ascontiguousarray(q[:, :2])
    sub_k = np.ascontiguousarray(k[:, :2])
    _softmax_check(mx, sub_q, sub_k, 75600 - 70, 70, "720p last rows")


def _diag_check(mx, P, N, mode, gamma, label):
    t = torch.from_numpy(np.ascontiguousarray(P, dtype=np.float32)).cuda()
    got = mx.rowsum_diag(t, N, mode, gamma).cpu().numpy()
    ref = oracle.rowsum_diag(P, N, MODES[mode], gamma)
    d = np.abs(got - ref)
    assert np.all(d[:, :7] <= 1e-11), f"{label}: worst {d[:, :7].max():.3g} at {np.unravel_index(d[:, :7].argmax(), d[:, :7].shape)}"
    assert np.all(d[:, 7] <= 1e-6 * ref[:, 7] + 1e-9), f"{label}: entropy {d[:, 7].max():.3g}"
    log(f"[rowsum diag] {label}: worst |diff| {d[:, :7].max():.3g}, entropy {d[:, 7].max():.3g}")
    return got


def _random_rows(seed, rows, N, spread):
    rng = np.random.default_rng(seed)
    s = rng.standard_normal((rows, N)) * spread
    P = np.exp(s - s.max(axis=1, keepdims=True))
    return (P / P.sum(axis=1, keepdims=True)).astype(np.float32)


@pytest.mark.parametrize("mode", list(MODES))
@pytest.mark.parametrize("gamma", [1.0, 2.0, 1.37])
def test_rowsum_diag_random_rows(mx, mode, gamma):
    for spread in (0.5, 2.0, 8.0):
        P = _random_rows(int(spread * 10), 300, 2048, spread)
        _diag_check(mx, P, 2048, mode, gamma, f"{mode} gamma={gamma} spread={spread}")


@pytest.mark.parametrize("mode", list(MODES))
def test_rowsum_diag_ragged_and_special_rows(mx, mode):
    N, ld = 1001, 1040
    P = np.full((8, ld), 0.7, np.float32)       # junk past N must be ignored
    P[:, :N] = _random_rows(7, 8, N, 3.0)
    P[1, :N] = np.float32(1.0) / np.float32(N)  # uniform
    P[2, :N] = 0.0
    P[2, 500] = 1.0                              # one-hot
    P[3, :N] = 0.0                               # empty
    P[4, :N] *= np.float32(2.0 ** -20)           # tiny values, normal fp32
    P[5, 10:40] = np.float32(3e-39)              # subnormal probabilities (entropy terms)
    P[5, 300] = np.float32(1e-44)
    got = _diag_check(mx, P, N, mode, 1.0, f"{mode} ragged/special")
    assert got[2, 0] == 1.0 and got[3, 0] == 0.0


def test_rowsum_diag_720p_rows_of_p(mx):
    """The GPU's own 720p probabilities, diagnosed on both sides."""
    q, k, _ = workload_bits(3)
    sub_q = np.ascontiguousarray(q[:, :1])
    sub_k = np.ascontiguousarray(k[:, :1])
    P = mx.softmax_rows(mx.bf16_from_bits(sub_q), mx.bf16_from_bits(sub_k), 1000, 64).cpu().numpy()
    P = P.reshape(64, -1)
    for mode in MODES:
        _diag_check(mx, P, 75600, mode, 1.0, f"720p {mode}")


def _same_stats(a, b, label):
    d = np.abs(a - b)
    assert np.all(d[..., :7] <= 1e-11), f"{label}: worst {d[..., :7].max():.3g}"
    assert np.all(d[..., 7] <= 1e-12 * np.abs(b[..., 7]) + 1e-12), f"{label}: entropy {d[..., 7].max():.3g}"
    log(f"[rowsum fused] {label}: worst |diff| {d[..., :7].max():.3g}")


@pytest.mark.parametrize("cfg", [0, 1])
def test_fused_diag_equals_composition(mx, cfg):
    q, k, _ = workload_bits(cfg)
    qt, kt = mx.bf16_from_bits(q), mx.bf16_from_bits(k)
    N = q.shape[2]
    for mode in MODES:
        for gamma in (1.0, 1.37):
            fused = mx.attention_rowsum_diag(qt, kt, mode, gamma).cpu().numpy()
            P = mx.softmax_rows(qt, kt)
            two = mx.rowsum_diag(P, N, mode, gamma).cpu().numpy().reshape(fused.shape)
            _same_stats(fused, two, f"cfg {cfg} {mode} gamma={gamma}")


def test_fused_diag_cross_lengths(mx):
    w = inputs.custom(1, 3, 700, kind="video", index=33)
    q, k, _ = inputs.generate(w)
    qt = mx.bf16_from_bits(np.ascontiguousarray(q[:, :, :130]))
    kt = mx.bf16_from_bits(np.ascontiguousarray(k[:, :, :700 - 3]))
    fused = mx.attention_rowsum_diag(qt, kt, "uos").cpu().numpy()
    P = mx.softmax_rows(qt, kt)
    two = mx.rowsum_diag(P, 697, "uos").cpu().numpy().reshape(fused.shape)
    _same_stats(fused, two, "Nq=130 Nkv=697")


def test_fused_diag_720p_sampled_rows(mx):
    """Whole 720p tensor diagnosed in one launch; sampled rows equal the
    diagnostic of the same rows materialized."""
    q, k, _ = workload_bits(3)
    qt, kt = mx.bf16_from_bits(q), mx.bf16_from_bits(k)
    fused = mx.attention_rowsum_diag(qt, kt, "uos").cpu().numpy()
    assert np.all(np.isfinite(fused))
    for row0 in (0, 37_000, 75600 - 40):
        P = mx.softmax_rows(qt, kt, row0, 40)
        part = mx.rowsum_diag(P, 75600, "uos").cpu().numpy().reshape(1, 40, 40, 8)
        _same_stats(fused[:, :, row0:row0 + 40], part, f"720p rows {row0}..")
        del P
    torch.cuda.empty_cache()


def test_report_rowsum_statistics(mx):
    """Mean row sum, its split and the entropy dependence (Fig. pnq_rowsum)
    on the synthetic workloads (logged)."""
    for cfg in (0, 1, 2, 3):
        w = inputs.workload(cfg)
        q, k, _ = workload_bits(cfg)
        qt, kt = mx.bf16_from_bits(q), mx.bf16_from_bits(k)
        for mode in MODES:
            st = mx.attention_rowsum_diag(qt, kt, mode).cpu().numpy().reshape(-1, 8)
            hi = st[:, 7] > 5.0
            log(f"[rowsum report] {w.name} {mode}: mean row sum {st[:, 0].mean():.4f} "
                f"(min {st[:, 0].min():.4f}, max {st[:, 0].max():.4f}); zeroing {st[:, 2].mean():+.4f} "
                f"saturation {st[:, 3].mean():+.4f} down {st[:, 4].mean():+.4f} up {st[:, 5].mean():+.4f}; "
                f"entropy > 5: {100 * hi.mean():.1f}% of rows, mean row sum there "
                f"{st[hi, 0].mean() if hi.any() else float('nan'):.4f}, below 1: "
                f"{100 * (st[hi, 0] < 1).mean() if hi.any() else float('nan'):.1f}%")
            assert np.allclose(st[:, 0] - st[:, 1], st[:, 2:7].sum(axis=1), atol=1e-12)
        torch.cuda.empty_cache()


def test_report_global_prescale(mx):
    """Fig. pnq_rowsum (C): one pre-quantization factor gamma for the whole
    tensor.  With power-of-two shared scales only the fraction of log2 gamma
    matters, so gamma runs over one octave (logged)."""
    for cfg in (1, 2):
        w = inputs.workload(cfg)
        q, k, _ = workload_bits(cfg)
        qt, kt = mx.bf16_from_bits(q), mx.bf16_from_bits(k)
        for mode in MODES:
            parts = []
            for i in range(8):
                gamma = 2.0 ** (i / 8)
                st = mx.attention_rowsum_diag(qt, kt, mode, gamma).cpu().numpy().reshape(-1, 8)
                parts.append(f"{gamma:.3f}: {st[:, 0].mean():.4f}/{100 * (st[:, 0] > 1).mean():.0f}%")
                if i == 0:  # gamma = 2 quantizes the same values (subnormal p aside)
                    np.testing.assert_allclose(
                        st, mx.attention_rowsum_diag(qt, kt, mode, 2.0).cpu().numpy().reshape(-1, 8),
                        rtol=0, atol=1e-20)
            log(f"[rowsum prescale] {w.name} {mode} (gamma: mean row sum / rows above 1): " + ", ".join(parts))
        torch.cuda.empty_cache()
