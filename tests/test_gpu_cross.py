"""Cross-attention on the GPU: Nq queries over Nkv keys/values (Wan2.2-style
video queries attending to a short text context, Sec. 5.1).

Output against the oracle fed the GPU's own codes (same tolerance as
self-attention), for ragged query and key lengths, every mode; the forward
equals attend() on separately quantized operands; with Nq = Nkv the cross
entry points equal the self-attention ones.  Up to 512 keys the K^/V^ of a
head stay resident in LDS and a workgroup runs several query tiles: lengths
on both sides of 512 and a case with two query tiles per workgroup and a
lone last one are covered.
"""
import numpy as np
import pytest

import oracle
from parity import MAX_ABS_TOL, REL_L2_TOL, flat, log, max_abs, oracle_rows, rel_l2, sample_rows
from paper_2607_24377_amd import inputs

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
MODES = ["ocp_vanilla", "uos", "uos_pnq", "uos_pnq_rot"]


@pytest.fixture(scope="module")
def mx():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_24377_amd import mxattn

    mxattn.lib()
    return mxattn


def _check(mx, w, mode, heads, n_rows, label):
    q, k, v = inputs.generate(w)
    qt, kt, vt = (mx.bf16_from_bits(x) for x in (q, k, v))
    out = mx.cross_forward(qt, kt, vt, mode)
    qc, qs = mx.quantize(qt, mx.AXIS_HEAD_DIM, mode)
    kc, ks = mx.quantize(kt, mx.AXIS_HEAD_DIM, mode)
    vc, vs = mx.quantize(vt, mx.AXIS_TOKENS, mode)
    again = mx.cross_attend(qc, qs, kc, ks, vc, vs, w.N, w.n_kv, mode)
    assert torch.equal(out, again)
    codes = {n: flat(t.cpu().numpy()) for n, t in dict(qc=qc, qs=qs, kc=kc, ks=ks, vc=vc, vs=vs).items()}
    got_all = flat(mx.bits_from_bf16(out))
    gots, refs = [], []
    for h in heads:
        rows = np.arange(w.N) if n_rows is None else sample_rows(w.N, n_rows, 500 + h)
        ref, _ = oracle_rows(codes, h, w.n_kv, rows, mode, mx.kv_tile())
        gots.append(oracle.bf16_to_f64(got_all[h][rows]))
        refs.append(ref)
    g, r = np.concatenate(gots), np.concatenate(refs)
    rl, ma = rel_l2(g, r), max_abs(g, r)
    log(f"[cross] {label} mode={mode}: rel-L2 {rl:.3e} max-abs {ma:.3e}")
    assert np.all(np.isfinite(g))
    assert rl <= REL_L2_TOL and ma <= MAX_ABS_TOL


@pytest.mark.parametrize("mode", MODES)
def test_cross_ragged_all_rows(mx, mode):
    w = inputs.workload("cross_ragged")
    _check(mx, w, mode, range(w.B * w.H), None, w.name)


@pytest.mark.parametrize("Nq,Nkv", [(200, 1), (200, 31), (1, 200), (129, 32), (130, 33), (300, 128),
                                    (64, 129), (257, 255), (130, 257), (200, 384), (300, 512),
                                    (300, 513), (130, 640), (64, 1100)])
def test_cross_ragged_lengths(mx, Nq, Nkv):
    w = inputs.Workload(60 + Nkv % 5, f"cross_{Nq}x{Nkv}", 2, 2, Nq, 128, "cross", Nkv=Nkv)
    for mode in ("ocp_vanilla", "uos_pnq"):
        _check(mx, w, mode, range(4), None, w.name)


def test_cross720p_sampled(mx):
    w = inputs.workload("cross720p")
    for mode in ("ocp_vanilla", "uos_pnq"):
        _check(mx, w, mode, [0, 39], 32, w.name)
    torch.cuda.empty_cache()


def test_equal_lengths_match_self_attention(mx):
    w = inputs.custom(1, 2, 300, kind="video", index=9)
    q, k, v = (mx.bf16_from_bits(x) for x in inputs.generate(w))
    assert torch.equal(mx.cross_forward(q, k, v, "uos_pnq"), mx.forward(q, k, v, "uos_pnq"))


def test_resident_several_query_tiles_per_workgroup(mx):
    # 16 heads x 129 query tiles = 2064 tiles: two per workgroup, the last
    # workgroup of each head gets one
    w = inputs.Workload(71, "cross_16x16500x500", 1, 16, 16500, 128, "cross", Nkv=500)
    for mode in ("ocp_vanilla", "uos_pnq"):
        _check(mx, w, mode, [0, 7, 15], 40, w.name)
    torch.cuda.empty_cache()


def test_resident_staged_stores_several_query_tiles(mx):
    # up to two key tiles the output rows go through an LDS buffer that each
    # query tile of a workgroup reuses: 16 heads x 129 query tiles, two per
    # workgroup, 200 keys (a full and a partial tile)
    w = inputs.Workload(72, "cross_16x16500x200", 1, 16, 16500, 128, "cross", Nkv=200)
    for mode in ("ocp_vanilla", "uos_pnq"):
        _check(mx, w, mode, [0, 9, 15], 40, w.name)
    torch.cuda.empty_cache()
