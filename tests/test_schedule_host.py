"""The product's step schedule agrees with the oracle's reading."""
import itertools

import pytest

from oracle import schedule as oracle_schedule

zf = pytest.importorskip("paper_2505_12242_amd")


@pytest.mark.parametrize("R,S", list(itertools.product([1, 2, 3, 4, 5, 8, 16], [1, 2, 3, 4, 8])))
def test_same_schedule(R, S):
    for t in range(1, 70):
        a = zf.schedule(t, R, S)
        b = oracle_schedule(t, R, S)
        assert (a.refresh, a.step_in_interval, a.interval_end) == \
            (b.refresh, b.step_in_interval, b.interval_end), (t, R, S)


@pytest.mark.parametrize("R,S,W", list(itertools.product([1, 2, 3, 4, 8], [1, 2, 4], [0, 1, 3, 9])))
def test_same_schedule_with_warmup(R, S, W):
    for t in range(1, 50):
        a = zf.schedule(t, R, S, W)
        b = oracle_schedule(t, R, S, W)
        assert (a.refresh, a.step_in_interval, a.interval_end) == \
            (b.refresh, b.step_in_interval, b.interval_end), (t, R, S, W)
