"""Pins of the oracle's fixed Hadamard rotation R_H (Sec. 4.3, Algorithm 2:
Q^rot = Q R_H, K^rot = K R_H before quantization).

* R_H = H / sqrt(128) with H the Sylvester Hadamard matrix: the image of every
  basis vector is checked entry by entry against (-1)^popcount(i & j) times
  fp32(1/sqrt(128)), which fixes the ordering and the sign of each butterfly.
* The fp32 transform stays within its rounding bound of the fp64 matrix
  product, and applying it twice returns the input (H H = 128 I).
* Orthogonality: Q R_H (K R_H)^T = Q K^T, so unquantized attention is unchanged.
* Outlier suppression, the reason the paper rotates: on the outlier-channel
  workload the MXFP4 error of the score matrix is smaller with the rotation.
"""
import struct

import numpy as np
import pytest

import oracle
from paper_2607_24377_amd import inputs

D = 128
S32 = struct.unpack("<f", struct.pack("<I", 0x3DB504F3))[0]  # fp32(1/sqrt(128))


def _sylvester(n):
    i = np.arange(n)
    pc = np.vectorize(lambda x: bin(x).count("1"))(i[:, None] & i[None, :])
    return np.where(pc % 2 == 0, 1.0, -1.0)


def test_scale_constant_is_nearest_fp32():
    assert S32 == np.float32(1.0 / np.sqrt(128.0))
    assert abs(S32 - 1 / np.sqrt(128.0)) <= np.spacing(np.float32(S32)) / 2


def test_basis_vectors_give_sylvester_columns():
    H = _sylvester(D)
    y = oracle.hadamard_f32(np.eye(D, dtype=np.float32))
    expect = (H * np.float64(S32)).astype(np.float32)
    assert np.array_equal(y, expect)


def test_fp32_transform_within_rounding_bound_of_fp64_product():
    rng = np.random.default_rng(3)
    x = rng.standard_normal((64, D)).astype(np.float32)
    x[:, [5, 77]] *= 300.0  # outlier channels
    y32 = oracle.hadamard_f32(x).astype(np.float64)
    y64 = x.astype(np.float64) @ _sylvester(D) / np.sqrt(D)
    bound = 9 * 2.0**-24 * np.abs(x.astype(np.float64)).sum(axis=1, keepdims=True) / np.sqrt(D)
    assert np.all(np.abs(y32 - y64) <= bound)


def test_transform_is_an_involution():
    rng = np.random.default_rng(4)
    x = rng.standard_normal((16, D)).astype(np.float32)
    back = oracle.hadamard_f32(oracle.hadamard_f32(x))
    np.testing.assert_allclose(back, x, rtol=0, atol=2e-6 * np.abs(x).max())


def test_rotation_preserves_scores_and_exact_attention():
    w = inputs.custom(1, 1, 256, kind="video", index=7)
    q, k, v = (oracle.bf16_to_f64(x[0, 0]) for x in inputs.generate(w))
    qr = oracle.hadamard_f32(q.astype(np.float32)).astype(np.float64)
    kr = oracle.hadamard_f32(k.astype(np.float32)).astype(np.float64)
    s, sr = q @ k.T, qr @ kr.T
    assert np.abs(sr - s).max() <= 1e-5 * np.abs(s).max()
    o = oracle.attention_exact_rows(q[:32], k, v)
    orot = oracle.attention_exact_rows(qr[:32], kr, v)
    np.testing.assert_allclose(orot, o, rtol=0, atol=1e-4)


def test_rotation_reduces_score_error_on_outlier_channels():
    w = inputs.workload("outlier_channels")
    q_bits, k_bits, _ = inputs.generate(w, heads=[0])
    q_bits, k_bits = q_bits[0, :512], k_bits[0, :512]
    q, k = oracle.bf16_to_f64(q_bits), oracle.bf16_to_f64(k_bits)
    s = q @ k.T
    err = {}
    for rot in (False, True):
        qc, qs = oracle.quantize_rows(q_bits, oracle.RULE_UOS, rotate=rot)
        kc, ks = oracle.quantize_rows(k_bits, oracle.RULE_UOS, rotate=rot)
        sh = oracle.dequant_rows(qc, qs) @ oracle.dequant_rows(kc, ks).T
        err[rot] = np.linalg.norm(sh - s) / np.linalg.norm(s)
    assert err[True] < 0.8 * err[False]


def test_rotated_quantizer_quantizes_the_rotated_rows():
    """The rotated quantizer = the block quantizer applied to hadamard_f32 rows
    (consistency of the two oracle entry points, not an independent pin)."""
    rng = np.random.default_rng(5)
    x = inputs.f32_to_bf16_bits(rng.standard_t(4, (8, D)).astype(np.float32))
    codes, scales = oracle.quantize_rows(x, oracle.RULE_UOS, rotate=True)
    y = oracle.hadamard_f32(oracle.bf16_to_f64(x).astype(np.float32)).astype(np.float64)
    for r in range(8):
        for b in range(4):
            c, sc = oracle.quantize_block(y[r, 32 * b:32 * b + 32], oracle.RULE_UOS)
            assert sc == scales[r, b]
            packed = c[0::2] | (c[1::2] << 4)
            assert np.array_equal(packed, codes[r, 16 * b:16 * b + 16])


@pytest.mark.parametrize("mode", ["uos_pnq_rot"])
def test_rotated_mode_quantizes_q_and_k_only(mode):
    w = inputs.custom(1, 1, 64, kind="iid", index=3)
    q, k, v = inputs.generate(w)
    got = oracle.quantize_qkv(q, k, v, mode)
    ref = oracle.quantize_qkv(q, k, v, "uos_pnq")
    assert not np.array_equal(got["qc"], ref["qc"])
    assert np.array_equal(got["vc"], ref["vc"]) and np.array_equal(got["vs"], ref["vs"])
