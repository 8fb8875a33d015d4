"""Suffix-wave sizing (paper Sec. 4.2): host logic, CPU only."""
import itertools

import pytest

from paper_2606_01143_amd.group import plan_suffix_waves


def _cost(lens, a, b, layout):
    return sum(lens[a:b]) if layout == "packed" else (b - a) * max(lens[a:b])


@pytest.mark.parametrize("layout", ["packed", "padded"])
@pytest.mark.parametrize("lens,budget", [((512,) * 8, 1024), ((128, 2048, 300, 900, 64, 1500), 2048),
                                         ((5, 1, 9, 3, 3, 7, 2), 10), ((100,), 50), ((3, 3, 3), 1000)])
def test_waves_cover_in_order_within_budget_and_greedy(lens, budget, layout):
    waves = plan_suffix_waves(lens, budget, layout)
    assert waves[0][0] == 0 and waves[-1][1] == len(lens)
    assert all(w1[1] == w2[0] for w1, w2 in zip(waves, waves[1:]))
    for a, b in waves:
        assert b > a
        assert _cost(lens, a, b, layout) <= budget or b == a + 1  # oversize suffixes alone
        if b < len(lens):
            assert _cost(lens, a, b + 1, layout) > budget  # greedy: the next one did not fit


def test_padded_waves_count_padding():
    # one long suffix makes the padded footprint large
    lens = (100, 100, 1000, 100)
    assert plan_suffix_waves(lens, 1100, "packed") == [(0, 2), (2, 4)]
    assert plan_suffix_waves(lens, 1100, "padded") == [(0, 2), (2, 3), (3, 4)]


def test_bad_arguments():
    with pytest.raises(ValueError):
        plan_suffix_waves((1, 2), 0)
    with pytest.raises(ValueError):
        plan_suffix_waves((1, 2), 10, "ragged")
