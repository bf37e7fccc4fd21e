"""The rotated mode on the GPU (Q and K multiplied by R_H = H/sqrt(128)
before MXFP4 quantization; Sec. 4.3, Algorithm 2).

* Q/K codes and scales bit-exact against the oracle's fp32 fast Walsh-Hadamard
  transform + block quantizer: random rows over a wide range of magnitudes,
  all-zero rows, and every element of Q and K of all five workloads.
* Attention output against the oracle fed the GPU's own (rotated) codes, to
  the usual tolerance; the forward equals attend() on separately quantized
  operands.
"""
import numpy as np
import pytest

import oracle
from parity import (MAX_ABS_TOL, REL_L2_TOL, flat, log, max_abs, oracle_rows, rel_l2, sample_rows,
                    workload_bits)
from paper_2607_24377_amd import inputs

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
MODE = "uos_pnq_rot"


@pytest.fixture(scope="module")
def mx():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_24377_amd import mxattn

    mxattn.lib()
    return mxattn


def _check_codes(mx, x, label):
    codes, scales = mx.quantize(mx.bf16_from_bits(x), mx.AXIS_HEAD_DIM, MODE)
    oc, os_ = oracle.quantize_rows(x, oracle.RULE_UOS, rotate=True)
    gs, gc = scales.cpu().numpy(), codes.cpu().numpy()
    assert np.array_equal(gs, os_), f"{label}: scales differ at {np.argwhere(gs != os_)[:5]}"
    assert np.array_equal(gc, oc), f"{label}: codes differ at {np.argwhere(gc != oc)[:5]}"


def test_random_rows_bit_exact(mx):
    rng = np.random.default_rng(11)
    rows = 8192
    mag = np.exp2(rng.integers(-100, 100, size=(rows, 1))).astype(np.float32)
    x = rng.standard_t(3, (rows, 128)).astype(np.float32) * mag
    x[rng.random((rows, 128)) < 0.05] *= 64.0  # sparse outliers
    x[::97] = 0.0                              # all-zero rows
    x[1::89, 3:] = 0.0                         # rows with few nonzeros
    bits = inputs.f32_to_bf16_bits(x).reshape(1, 1, rows, 128)
    log("[rot codes] random rows")
    _check_codes(mx, bits, "random rows")


@pytest.mark.parametrize("cfg", [0, 1, 2, 3, 4])
def test_workload_codes_bit_exact(mx, cfg):
    q, k, _ = workload_bits(cfg)
    w = inputs.workload(cfg)
    for name, x in (("q", q), ("k", k)):
        log(f"[rot codes] {w.name} {name}")
        _check_codes(mx, x, f"{w.name} {name}")
    torch.cuda.empty_cache()


def _attention_rows(mx, cfg, heads, n_rows):
    w = inputs.workload(cfg)
    q, k, v = workload_bits(cfg)
    qt, kt, vt = (mx.bf16_from_bits(x) for x in (q, k, v))
    out = flat(mx.bits_from_bf16(mx.forward(qt, kt, vt, MODE)))
    qc, qs = mx.quantize(qt, mx.AXIS_HEAD_DIM, MODE)
    kc, ks = mx.quantize(kt, mx.AXIS_HEAD_DIM, MODE)
    vc, vs = mx.quantize(vt, mx.AXIS_TOKENS, MODE)
    codes = {n: flat(t.cpu().numpy()) for n, t in dict(qc=qc, qs=qs, kc=kc, ks=ks, vc=vc, vs=vs).items()}
    gots, refs = [], []
    for h in heads:
        rows = np.arange(w.N) if n_rows is None else sample_rows(w.N, n_rows, 300 + h, w.text_tokens)
        ref, _ = oracle_rows(codes, h, w.N, rows, MODE, mx.kv_tile())
        gots.append(oracle.bf16_to_f64(out[h][rows]))
        refs.append(ref)
    g, r = np.concatenate(gots), np.concatenate(refs)
    rl, ma = rel_l2(g, r), max_abs(g, r)
    log(f"[rot attn] {w.name}: rel-L2 {rl:.3e} max-abs {ma:.3e}")
    assert np.all(np.isfinite(g))
    assert rl <= REL_L2_TOL and ma <= MAX_ABS_TOL
    # the forward equals attend() on the separately quantized operands
    again = mx.attend(qc, qs, kc, ks, vc, vs, w.N, MODE)
    assert torch.equal(mx.forward(qt, kt, vt, MODE), again)


def test_attention_tiny_all_rows(mx):
    _attention_rows(mx, 0, [0, 1], None)


def test_attention_outlier_channels_sampled(mx):
    _attention_rows(mx, 1, [0, 21, 39], 48)


def test_attention_joint_text_video_sampled(mx):
    _attention_rows(mx, 4, [0, 23], 24)
