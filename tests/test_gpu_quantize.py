"""GPU quantizer vs the CPU oracle: codes and E8M0 scales bit-exact.

* every finite bf16 value (next to fixed anchors) through both block axes;
* every element of Q, K (blocks along d) and V (blocks along tokens) of all
  five workloads under both scale rules.
"""
import numpy as np
import pytest

import oracle
from parity import log, workload_bits
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


RULE = {"ocp_vanilla": oracle.RULE_OCP, "uos": oracle.RULE_UOS}


def _finite_bf16():
    b = np.arange(65536, dtype=np.uint32).astype(np.uint16)
    return b[((b >> 7) & 0xFF) != 0xFF]


@pytest.mark.parametrize("mode", ["ocp_vanilla", "uos"])
@pytest.mark.parametrize("anchor", [0.0, 1.0, 6.0, 6.0 * 2.0**-40, 6.0 * 2.0**40, 2.0**-133,
                                    2.0**-126, 7.25 * 2.0**-128])
def test_exhaustive_bf16_head_dim(mx, mode, anchor):
    log(f"[quant exhaustive head-dim] mode={mode} anchor={anchor}")
    bits = _finite_bf16()
    n = bits.size
    x = np.zeros((n, 32), dtype=np.uint16)
    x[:, 0] = bits
    x[:, 17] = inputs.f32_to_bf16_bits(np.full(n, anchor, np.float32))
    x[:, 31] = bits[::-1]
    # 4 blocks per 128-wide row
    pad = (-n) % 4
    xx = np.concatenate([x, np.zeros((pad, 32), np.uint16)]).reshape(1, 1, -1, 128)
    codes, scales = mx.quantize(mx.bf16_from_bits(xx), mx.AXIS_HEAD_DIM, mode)
    oc, os_ = oracle.quantize_rows(xx, RULE[mode])
    np.testing.assert_array_equal(scales.cpu().numpy(), os_)
    np.testing.assert_array_equal(codes.cpu().numpy(), oc)


@pytest.mark.parametrize("mode", ["ocp_vanilla", "uos"])
@pytest.mark.parametrize("anchor", [0.0, 6.0, 2.0**-133, 6.0 * 2.0**40])
def test_exhaustive_bf16_tokens(mx, mode, anchor):
    """The same sweep with blocks running along the token axis; N is not a
    multiple of 32 so the zero-padded tail block is exercised too."""
    log(f"[quant exhaustive tokens] mode={mode} anchor={anchor}")
    bits = _finite_bf16()
    N = 32 * 16 + 19
    total = bits.size
    n_heads = -(-total // (N * 128))
    flat = np.zeros(n_heads * N * 128, dtype=np.uint16)
    flat[:total] = bits
    x = flat.reshape(n_heads, N, 128)
    x[:, 5, :] = inputs.f32_to_bf16_bits(np.full((n_heads, 128), anchor, np.float32))
    x = x.reshape(1, n_heads, N, 128)
    codes, scales = mx.quantize(mx.bf16_from_bits(x), mx.AXIS_TOKENS, mode)
    oc, os_ = oracle.quantize_keys(x, RULE[mode])
    np.testing.assert_array_equal(scales.cpu().numpy(), os_)
    np.testing.assert_array_equal(codes.cpu().numpy(), oc)


@pytest.mark.parametrize("cfg", [0, 1, 2, 3, 4])
def test_workload_codes_bit_exact(mx, cfg):
    q, k, v = workload_bits(cfg)
    w = inputs.workload(cfg)
    for mode in ("ocp_vanilla", "uos"):
        log(f"[quant workload] {w.name} mode={mode}")
        for name, x, axis in (("q", q, mx.AXIS_HEAD_DIM), ("k", k, mx.AXIS_HEAD_DIM),
                              ("v", v, mx.AXIS_TOKENS)):
            xt = mx.bf16_from_bits(x)
            codes, scales = mx.quantize(xt, axis, mode)
            if axis == mx.AXIS_HEAD_DIM:
                oc, os_ = oracle.quantize_rows(x, RULE[mode])
            else:
                oc, os_ = oracle.quantize_keys(x, RULE[mode])
            gs = scales.cpu().numpy()
            gc = codes.cpu().numpy()
            assert np.array_equal(gs, os_), f"{name} scales differ at {np.argwhere(gs != os_)[:5]}"
            assert np.array_equal(gc, oc), f"{name} codes differ at {np.argwhere(gc != oc)[:5]}"
            del xt, codes, scales
        torch.cuda.empty_cache()
