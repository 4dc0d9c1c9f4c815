"""Pins the step schedule: refresh / interval start / interval end."""
import itertools

import pytest

from oracle import schedule


def table(R, S, T):
    return [schedule(t, R, S) for t in range(1, T + 1)]


def test_refresh_equals_interval():
    ks = table(4, 4, 16)
    assert [t for t, k in enumerate(ks, 1) if k.refresh] == [1, 5, 9, 13]
    assert [k.step_in_interval for k in ks] == [1, 2, 3, 4] * 4
    assert [t for t, k in enumerate(ks, 1) if k.interval_end] == [4, 8, 12, 16]


def test_refresh_every_step_forces_unit_intervals():
    for k in table(1, 4, 10):
        assert k.refresh and k.step_in_interval == 1 and k.interval_end


def test_slow_refresh():
    ks = table(16, 4, 20)
    assert [t for t, k in enumerate(ks, 1) if k.refresh] == [1, 17]
    assert [t for t, k in enumerate(ks, 1) if k.interval_end] == [4, 8, 12, 16, 20]


def test_unaligned_refresh_cuts_intervals():
    ks = table(3, 4, 12)
    assert [k.step_in_interval for k in ks] == [1, 2, 3, 1, 1, 2, 1, 2, 1, 1, 2, 3]


@pytest.mark.parametrize("R,S", list(itertools.product(range(1, 7), range(1, 7))))
def test_consistency(R, S):
    ks = table(R, S, 60)
    nxt = schedule(61, R, S)
    for t, k in enumerate(ks, 1):
        following = ks[t] if t < 60 else nxt
        assert k.interval_end == (following.step_in_interval == 1)
        if k.refresh:
            assert k.step_in_interval == 1
        if t > 1 and k.step_in_interval > 1:
            assert ks[t - 2].step_in_interval == k.step_in_interval - 1
        assert 1 <= k.step_in_interval <= S


def test_bad_arguments():
    for args in [(0, 4, 4), (1, 0, 4), (1, 4, 0)]:
        with pytest.raises(ValueError):
            schedule(*args)


def test_warmup_zero_is_the_plain_schedule():
    for R, S in itertools.product(range(1, 7), range(1, 7)):
        for t in range(1, 40):
            assert schedule(t, R, S, 0) == schedule(t, R, S)


def test_warmup_table():
    """tau = 3, R = 8, S = 4: one-step intervals at t = 1..3, then S-step
    intervals counted from t = 4 (4..7, 8), cut by the refresh at 9."""
    ks = [schedule(t, 8, 4, 3) for t in range(1, 14)]
    assert [t for t, k in enumerate(ks, 1) if k.interval_end] == [1, 2, 3, 7, 8, 11]
    assert [k.step_in_interval for k in ks] == [1, 1, 1, 1, 2, 3, 4, 1, 1, 2, 3, 1, 2]
    assert [t for t, k in enumerate(ks, 1) if k.refresh] == [1, 9]


def test_warmup_longer_than_the_run_hands_over_every_step():
    for k in (schedule(t, 4, 4, 50) for t in range(1, 51)):
        assert k.step_in_interval == 1 and k.interval_end


@pytest.mark.parametrize("R,S,W", list(itertools.product([1, 2, 4, 7], [1, 3, 4], [0, 1, 5])))
def test_warmup_consistency(R, S, W):
    """Lengths increase by one inside an interval and restart at 1 right
    after every end; an interval never exceeds S steps after the warm-up and
    one step within it."""
    prev_end = True
    for t in range(1, 40):
        k = schedule(t, R, S, W)
        assert k.step_in_interval == (1 if prev_end else prev_len + 1)
        assert k.step_in_interval <= (1 if t <= W else S)
        prev_end, prev_len = k.interval_end, k.step_in_interval
