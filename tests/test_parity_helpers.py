"""Host logic of the GPU parity tests (no GPU): the stratified row sample and
the acceptance of bf16 rounding ties."""
import numpy as np

from parity import BF16_TIE_WINDOW, bf16_ties, stratified_rows


def test_bf16_ties_accepts_only_neighbours_at_a_midpoint():
    # 2.984375 and 3.0 are neighbouring bf16 values (ulp 2^-6 in [2, 4))
    lo, hi = 2.984375, 3.0
    mid = 0.5 * (lo + hi)
    got = np.array([hi, hi, hi, lo, 3.015625, 1.0])
    ref = np.array([lo, lo, lo, hi, lo, 1.0])
    x = np.array([mid * (1 - 0.5 * BF16_TIE_WINDOW),   # within the window
                  mid * (1 - 2.0 * BF16_TIE_WINDOW),   # outside it
                  lo,                                  # exactly representable: one valid rounding
                  mid * (1 + 0.25 * BF16_TIE_WINDOW),  # within, other side
                  2.999,                               # not neighbours (two ulps apart)
                  1.0])                                # equal: not a tie
    np.testing.assert_array_equal(bf16_ties(got, ref, x), [True, False, False, True, False, False])
    # negative values
    assert bf16_ties(np.array([-hi]), np.array([-lo]), np.array([-mid]))[0]


def test_stratified_rows_cover_edges_text_and_heads():
    N, H, text = 119056, 24, 256
    rows = {h: stratified_rows(N, h, H, 86, 7 + h, text) for h in range(H)}
    for h, r in rows.items():
        assert r.size >= 86 and np.all(np.diff(r) > 0) and r[0] == 0 and r[-1] == N - 1
        assert (N - 1) // 128 * 128 in r  # first row of the ragged last query tile
        assert {1, 63, 127} <= set(r.tolist())
    covered = set().union(*(set(r.tolist()) & set(range(N - text, N)) for r in rows.values()))
    assert covered == set(range(N - text, N))  # every text row, over the heads
    small = stratified_rows(40, 0, 2, 1024, 0)
    np.testing.assert_array_equal(small, np.arange(40))  # short sequences: every row
