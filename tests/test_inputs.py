"""The seeded synthetic workloads: determinism, per-head regeneration and the
distribution recipe of each workload."""
import numpy as np

from paper_2607_24377_amd import inputs


def test_deterministic_and_per_head():
    w = inputs.custom(1, 3, 100, kind="video")
    a = inputs.generate(w)
    b = inputs.generate(w)
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x, y)
    one = inputs.generate(w, heads=[2])
    for x, y in zip(a, one):
        np.testing.assert_array_equal(x[0, 2], y[0])


def test_bf16_rounding_is_nearest_even():
    x = np.array([1.0, 1.00390625, 1.01171875, -2.5, 3.0e38], dtype=np.float32)
    bits = inputs.f32_to_bf16_bits(x)
    back = inputs.bf16_bits_to_f32(bits)
    np.testing.assert_array_equal(back[:2], [1.0, 1.0])       # tie -> even
    assert back[2] == np.float32(1.015625)                      # tie -> even (up)
    assert back[3] == -2.5


def test_workload_shapes_and_flops():
    w = inputs.workload("video720p")
    assert (w.B, w.H, w.N, w.d) == (1, 40, 75600, 128)
    assert abs(w.flops - 117.05e12) / 117.05e12 < 1e-3
    assert inputs.workload(4).N == 33 * 45 * 80 + 256
    assert inputs.workload(2).N == 21 * 30 * 52


def test_distribution_recipes():
    w = inputs.custom(1, 2, 4096, kind="video", index=2)
    q, k, v = (inputs.bf16_bits_to_f32(t)[0] for t in inputs.generate(w))
    # Student-t(4) has variance 2; the K offset has variance 2 per channel
    assert abs(q.var() - 2.0) < 0.3
    mu = k.mean(axis=1)  # per (head, channel) means
    assert 0.8 < mu.var() < 4.0
    assert abs(v.std() - 1.0) < 0.02
    wo = inputs.custom(1, 2, 2048, kind="outlier", index=1)
    q, k, _ = (inputs.bf16_bits_to_f32(t)[0] for t in inputs.generate(wo))
    for h in range(2):
        big_q = set(np.argsort(q[h].std(axis=0))[-4:])
        big_k = set(np.argsort(k[h].std(axis=0))[-4:])
        assert big_q == big_k                      # shared outlier channels
        assert q[h].std(axis=0).max() > 15
    wt = inputs.custom(1, 1, 600, kind="video", text_tokens=256, index=4)
    q, k, v = (inputs.bf16_bits_to_f32(t)[0, 0] for t in inputs.generate(wt))
    assert np.abs(q[-256:]).mean() > 3 * np.abs(q[:-256]).mean()
    assert abs(np.abs(v[-256:]).mean() - np.abs(v[:-256]).mean()) < 0.1
