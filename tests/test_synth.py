"""The seeded input layer: budget layouts of the Appendix B strategies U, R
and F, group sizes, and determinism of the draws."""

import numpy as np
import pytest

import synth

GROUPS = ((40, 0.25), (20, 0.25), (10, 0.5))


@pytest.mark.parametrize("layout", ["scattered", "contiguous", "random", "uniform", "first_frame"])
def test_layouts_fill_the_group_sizes(layout):
    N = 32760
    v = np.random.default_rng(0).standard_normal((N, 4)).astype(np.float32)
    b = synth.assign_budgets(v, GROUPS, layout, frame_tokens=30 * 52, seed=5)
    assert [int((b == s).sum()) for s, _ in synth.group_sizes(N, GROUPS)] == [n for _, n in synth.group_sizes(N, GROUPS)]
    np.testing.assert_array_equal(b, synth.assign_budgets(v, GROUPS, layout, frame_tokens=30 * 52, seed=5))


def test_first_frame_reserved_for_the_largest_budget():
    N, frame = 21 * 30 * 52, 30 * 52
    b = synth.assign_budgets(np.zeros((N, 1), np.float32), GROUPS, "first_frame", frame_tokens=frame, seed=1)
    assert np.all(b[:frame] == 40)
    with pytest.raises(ValueError):
        synth.assign_budgets(np.zeros((100, 1), np.float32), GROUPS, "first_frame", frame_tokens=30, seed=1)


def test_uniform_groups_span_the_sequence():
    N = 32760
    b = synth.assign_budgets(np.zeros((N, 1), np.float32), GROUPS, "uniform")
    for s, n in synth.group_sizes(N, GROUPS):
        pos = np.flatnonzero(b == s)
        assert np.diff(pos).max() <= 2 * N / n  # no gap beyond twice the even spacing
        # every frame of 1560 tokens holds its share of the group, within 2%
        per_frame = np.bincount(pos // 1560, minlength=21)
        assert np.all(np.abs(per_frame - n / 21) <= 0.02 * 1560)


def test_random_budgets_seeded():
    a = synth.random_budgets(1000, GROUPS, seed=3)
    assert np.array_equal(a, synth.random_budgets(1000, GROUPS, seed=3))
    assert not np.array_equal(a, synth.random_budgets(1000, GROUPS, seed=4))
