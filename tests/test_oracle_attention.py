"""Pins of the oracle's tiled online-softmax attention.

* With the identity quantizer in fp64 the recurrence must equal textbook
  softmax attention (Eq. standard_attention), for any KV tile width.
* With MXFP4 quantization of P~, an independent numpy evaluation of the
  effective full-row form (App. "Full Online-Softmax Form of PNQ", Lemma
  pnq_effective_full_row: every tile rescaled by beta_j = exp(m_j - m_final))
  must equal the recurrence.
* Proposition 1: PNQ's induced weights sum to one; direct placement's do not
  (Eq. pnq_direct_full_rowsum).
* Special cases with closed forms: V = 1 and identical keys.
"""
import numpy as np
import pytest

import oracle

UOS, OCP, ID = oracle.RULE_UOS, oracle.RULE_OCP, oracle.RULE_IDENTITY
LOG2E = 1.4426950408889634


def _textbook(q, k, v):
    s = q @ k.T / np.sqrt(q.shape[1])
    s = s - s.max(axis=1, keepdims=True)
    p = np.exp(s)
    p /= p.sum(axis=1, keepdims=True)
    return p @ v


def _rand(R, N, d, seed, scale=1.0):
    rng = np.random.default_rng(seed)
    return (rng.standard_normal((R, d)) * scale, rng.standard_normal((N, d)) * scale,
            rng.standard_normal((N, d)))


@pytest.mark.parametrize("block_c", [1, 7, 32, 100, 128, 300, 1000])
def test_identity_quantizer_is_textbook_attention(block_c):
    q, k, v = _rand(9, 300, 64, 0, scale=1.5)
    out = oracle.attention_rows(q, k, v, ID, 0, exact=1, block_c=block_c)
    np.testing.assert_allclose(out, _textbook(q, k, v), rtol=0, atol=1e-12)
    out2 = oracle.attention_rows(q, k, v, ID, 1, exact=1, block_c=block_c)
    np.testing.assert_allclose(out2, out, rtol=0, atol=1e-13)
    ex = oracle.attention_exact_rows(q, k, v)
    np.testing.assert_allclose(ex, _textbook(q, k, v), rtol=0, atol=1e-12)


def _quantize_tile_numpy(p, rule):
    """P^ of one tile row by 32-key blocks (block quantizer from the oracle)."""
    out = np.zeros_like(p)
    for b in range(0, p.size, 32):
        seg = p[b:b + 32]
        codes, sc = oracle.quantize_block(seg, rule)
        out[b:b + seg.size] = [oracle.decode(int(c), sc) for c in codes]
    return out


def _effective_row_form(q, k, v, rule, pnq, block_c):
    """Independent evaluation in fp64: all scores at once, running maxima per
    tile, every tile's contribution rescaled by beta_j = 2^(m_j - m_final)."""
    R, d = q.shape
    N = k.shape[0]
    c = LOG2E / np.sqrt(d)
    s2 = (q @ k.T) * c
    out = np.zeros((R, d))
    rowsum = np.zeros(R)
    for r in range(R):
        tiles = [(j0, min(N, j0 + block_c)) for j0 in range(0, N, block_c)]
        m, ms = -np.inf, []
        for a, b in tiles:
            m = max(m, s2[r, a:b].max())
            ms.append(m)
        mfin = ms[-1]
        l = 0.0
        mass_hat = 0.0
        o = np.zeros(d)
        for (a, b), mj in zip(tiles, ms):
            pt = np.exp2(s2[r, a:b] - mj)
            padded = np.zeros(block_c)
            padded[:b - a] = pt
            ph = _quantize_tile_numpy(padded, rule)[:b - a]
            beta = np.exp2(mj - mfin)
            l += beta * (ph.sum() if pnq else pt.sum())
            mass_hat += beta * ph.sum()
            o += beta * (ph @ v[a:b])
        out[r] = o / l
        rowsum[r] = mass_hat / l
    return out, rowsum


@pytest.mark.parametrize("rule,pnq", [(OCP, 0), (UOS, 0), (UOS, 1)])
@pytest.mark.parametrize("N,block_c", [(200, 64), (77, 32), (256, 128), (129, 128)])
def test_recurrence_equals_effective_row_form(rule, pnq, N, block_c):
    q, k, v = _rand(6, N, 128, N + block_c, scale=1.2)
    out, dg = oracle.attention_rows(q, k, v, rule, pnq, exact=1, block_c=block_c, diag=True)
    ref, rowsum = _effective_row_form(q, k, v, rule, pnq, block_c)
    np.testing.assert_allclose(out, ref, rtol=0, atol=1e-12)
    np.testing.assert_allclose(dg[:, 1], rowsum, rtol=1e-12)
    # the oracle's own unrolled bookkeeping agrees with its recurrence
    assert np.all(dg[:, 3] < 1e-12)
    np.testing.assert_allclose(dg[:, 2], dg[:, 0], rtol=1e-12)


@pytest.mark.parametrize("exact", [0, 1])
def test_kernel_contract_close_to_fp64(exact):
    q, k, v = _rand(5, 200, 128, 11)
    out32 = oracle.attention_rows(q, k, v, UOS, 1, exact=0, block_c=64)
    ref, _ = _effective_row_form(q, k, v, UOS, 1, 64)
    # fp32 score/exp rounding only moves codes whose P~ sits at a threshold
    assert np.sqrt(np.sum((out32 - ref) ** 2) / np.sum(ref ** 2)) < 2e-3


def test_pnq_rows_sum_to_one_direct_rows_do_not():
    q, k, v = _rand(64, 2048, 128, 21)
    sums = {}
    for name, (rule, pnq) in oracle.MODES.items():
        _, dg = oracle.attention_rows(q, k, v, rule, pnq, exact=0, block_c=128, diag=True)
        sums[name] = dg[:, 1]
        assert np.all(dg[:, 3] < 1e-12)
    np.testing.assert_allclose(sums["uos_pnq"], 1.0, rtol=0, atol=1e-12)  # Proposition 1
    for name in ("ocp_vanilla", "uos"):
        assert np.max(np.abs(sums[name] - 1.0)) > 1e-3
        assert np.mean(sums[name]) < 1.0  # net loss of mass, as the paper observes


def test_v_all_ones():
    rng = np.random.default_rng(4)
    N, d = 300, 128
    ones = np.ones((1, N, d), dtype=np.float32)
    from paper_2607_24377_amd.inputs import f32_to_bf16_bits
    vc, vs = oracle.quantize_keys(f32_to_bf16_bits(ones), UOS)
    vh = oracle.dequant_keys(vc[0], vs[0], N)
    assert np.all(vh == 1.0)  # block max 1 -> e = -2 -> 4 on the grid
    q, k = rng.standard_normal((8, d)) * 2, rng.standard_normal((N, d)) * 2
    for name, (rule, pnq) in oracle.MODES.items():
        out, dg = oracle.attention_rows(q, k, vh, rule, pnq, exact=0, block_c=128, diag=True)
        np.testing.assert_allclose(out, np.repeat(dg[:, 1:2], d, axis=1), rtol=1e-13)
        if pnq:
            np.testing.assert_array_equal(oracle.round_bf16(out), 0x3F80)  # exactly 1.0


def test_identical_keys_average_values():
    rng = np.random.default_rng(6)
    N, d = 200, 128
    k = np.repeat(rng.standard_normal((1, d)), N, axis=0)
    q = rng.standard_normal((4, d))
    v = rng.standard_normal((N, d))
    for name, (rule, pnq) in oracle.MODES.items():
        for exact in (0, 1):
            out = oracle.attention_rows(q, k, v, rule, pnq, exact=exact, block_c=64)
            tol = 1e-12 if (pnq or exact) else 1e-6
            np.testing.assert_allclose(out, np.repeat(v.mean(0, keepdims=True), 4, 0),
                                       rtol=0, atol=tol)


def test_pnq_closes_gap_on_iid_data():
    """UOS+PNQ's least-squares gain against exact attention is nearer to one
    than vanilla OCP's (the direction the paper's ablation reports)."""
    rng = np.random.default_rng(8)
    N, d = 2048, 128
    from paper_2607_24377_amd.inputs import f32_to_bf16_bits
    x = f32_to_bf16_bits(rng.standard_normal((3, 1, N, d)).astype(np.float32))
    ref = oracle.attention_exact_rows(oracle.bf16_to_f64(x[0, 0, :64]), oracle.bf16_to_f64(x[1, 0]),
                                      oracle.bf16_to_f64(x[2, 0]))
    gains = {}
    for mode in oracle.MODES:
        qq = oracle.quantize_qkv(x[0][None], x[1][None], x[2][None], mode)
        out = oracle.mx_attention_head_rows(qq["qc"][0, 0], qq["qs"][0, 0], qq["kc"][0, 0],
                                            qq["ks"][0, 0], qq["vc"][0, 0], qq["vs"][0, 0], N,
                                            np.arange(64), mode)
        gains[mode] = float(np.sum(out * ref) / np.sum(ref * ref))
    assert abs(gains["uos_pnq"] - 1) < abs(gains["ocp_vanilla"] - 1)
    assert abs(gains["uos_pnq"] - 1) < 0.1


def _score_for(t: float, c32: np.float32) -> float:
    """An fp32 score s whose fp32 product with c32 is exactly t (float32)."""
    t32 = np.float32(t)
    s = np.float32(t32 / c32)
    for _ in range(64):
        p = np.float32(np.float64(s) * np.float64(c32))
        if p == t32:
            return float(s)
        s = np.nextafter(s, np.float32(np.inf) if p < t32 else np.float32(-np.inf))
    raise AssertionError("no fp32 score for t")


@pytest.mark.parametrize("rule,near_el,near_blk", [(UOS, 2, 1), (OCP, 2, 1)])
def test_exponential_audit_counts_planted_cases(rule, near_el, near_blk):
    """Diagnostic columns 6 and 7 count exactly the elements of P~ that sit
    within 4 fp32 ulps of an E2M1 decision threshold (App. B midpoints) and
    the blocks whose maximum sits within 4 ulps of an end of the scale
    rule's range.  One query (d = 1, so c = log2 e) against planted scores:
    block 0 holds the row maximum (t = 0, P~ = 1, sigma = 1/4 under both
    rules), P~ = 2^-4 (normalized 0.25, a tie) and P~ ~ 0.1875 (normalized
    0.75); block 1's maximum is ~ 7.25 * 2^-5 (the UOS boundary); block 2's is
    2^-3 (the OCP boundary 4 sigma).  Every other score has t = -10."""
    c32 = np.float32(1.4426950408889634)
    t = np.full(72, -10.0)
    t[0], t[1], t[2] = 0.0, -4.0, np.log2(0.1875)
    t[32] = np.log2(7.25 * 2.0 ** -5)
    t[64] = -3.0
    k = np.array([[_score_for(x, c32)] for x in t])
    q = np.ones((1, 1))
    v = np.ones((72, 1))
    _, dg = oracle.attention_rows(q, k, v, rule, 1, exact=0, block_c=128, diag=True)
    assert dg.shape == (1, 8)
    assert (dg[0, 6], dg[0, 7]) == (near_el, near_blk)
    # the unquantized path has nothing to audit
    _, dg = oracle.attention_rows(q, k, v, ID, 1, exact=0, block_c=128, diag=True)
    assert (dg[0, 6], dg[0, 7]) == (0, 0)
