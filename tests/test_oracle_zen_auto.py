"""Pins of the oracle's Zen-auto functions (adaptive accumulation interval,
Zero-stall Pipeline, "Hyperparameter Auto-tuning").

* column_sq_norms: n = 1 reduces to one correctly rounded fp32 square; dyadic
  columns have exact closed forms; the column norms add up to the squared
  Frobenius norm (numpy's fp64 norm).
* zen_auto_stats: slot order follows sel / unsel, on a hand-built matrix.
* zen_auto_trigger: exact dyadic examples, including the equality case, the
  pooled mean over matrices (not the mean of per-matrix means), empty parts.
* ZenAutoOracle: the worked example of the Sensitivity section (a channel at
  0.1 per step reaches 0.5 after five steps); tau = inf gives the fixed
  schedule with S = S_max bit for bit (R a multiple of S); tau = 0 gives
  intervals of one step; structural invariants of the schedule for
  intermediate tau.
"""
import math

import numpy as np
import pytest

import oracle as O


def bf16(x):
    return O.bf16_round(np.asarray(x, dtype=np.float32))


# ---------------------------------------------------------------- norms

def test_column_sq_norms_single_row_is_one_fp32_square():
    rng = np.random.default_rng(0)
    x = (rng.standard_normal(4096) * np.exp2(rng.integers(-80, 60, 4096))).astype(np.float32)
    got = O.column_sq_norms(x[None, :])
    want = x * x  # IEEE fp32 multiply: the exact square rounded once
    assert np.array_equal(got.view(np.uint32), want.view(np.uint32))


def test_column_sq_norms_dyadic_closed_form():
    n, m = 37, 12
    e = np.arange(m) - 6
    X = np.tile(np.exp2(e).astype(np.float32), (n, 1))
    X[::2] *= -1
    got = O.column_sq_norms(X)
    assert np.array_equal(got, (n * np.exp2(2.0 * e)).astype(np.float32))


def test_column_sq_norms_sum_to_frobenius():
    rng = np.random.default_rng(1)
    X = (rng.standard_normal((300, 77)) * np.exp(rng.standard_normal(77))).astype(np.float32)
    s = O.column_sq_norms(X).astype(np.float64)
    frob = np.linalg.norm(X.astype(np.float64)) ** 2
    assert abs(s.sum() - frob) <= 1e-6 * frob
    # and per column against numpy's fp64 vector norm (one fp32 rounding)
    ref = np.linalg.norm(X.astype(np.float64), axis=0) ** 2
    assert np.all(np.abs(s - ref) <= 2 ** -23 * ref)


def test_zen_auto_stats_slot_order():
    # 2 x 5 gradient, columns 1 and 3 selected; column j holds the value j+1
    G = bf16(np.tile(np.arange(1, 6, dtype=np.float32), (2, 1)))
    sel = O.select_topk(np.array([0, 5, 0, 7, 0], dtype=np.float32), 2)
    assert list(sel.sel) == [1, 3] and list(sel.unsel) == [0, 2, 4]
    A = np.array([[1, 2, 3], [1, 2, 3]], dtype=np.float32)  # packed slots 0..2
    sel_sq, acc_sq = O.zen_auto_stats(G, sel, A)
    assert list(sel_sq) == [2 * 4.0, 2 * 16.0]   # columns 1, 3 hold 2 and 4
    assert list(acc_sq) == [2.0, 8.0, 18.0]


# ---------------------------------------------------------------- trigger

def test_trigger_exact_example_and_boundary():
    stats = [(np.array([4.0, 4.0], np.float32), np.array([1.0, 1.0], np.float32))]
    # mean selected norm 2, mean accumulated norm 1 -> ratio exactly 1/2
    t = O.zen_auto_trigger(stats, 0.5)
    assert (t.sum_sel, t.k, t.sum_acc, t.u, t.trigger) == (4.0, 2, 2.0, 2, True)
    assert not O.zen_auto_trigger(stats, 0.5 + 2 ** -40).trigger
    assert O.zen_auto_trigger(stats, 0.25).trigger


def test_trigger_pools_channels_over_matrices():
    # matrix 1: one selected channel of norm 10, nine unselected of norm 1;
    # matrix 2: nine selected of norm 1, one unselected of norm 10.
    # pooled: mean sel = 19/10, mean acc = 19/10 -> ratio 1; the mean of the
    # per-matrix ratios would be (0.1 + 10) / 2.
    s1 = (np.array([100.0], np.float32), np.ones(9, np.float32))
    s2 = (np.ones(9, np.float32), np.array([100.0], np.float32))
    t = O.zen_auto_trigger([s1, s2], 1.0)
    assert (t.sum_sel, t.k, t.sum_acc, t.u) == (19.0, 10, 19.0, 10)
    assert t.trigger
    assert not O.zen_auto_trigger([s1, s2], 1.0 + 1e-12).trigger


def test_trigger_empty_parts():
    e = np.zeros(0, np.float32)
    assert not O.zen_auto_trigger([(e, np.ones(3, np.float32))], 0.0).trigger
    assert not O.zen_auto_trigger([(np.ones(3, np.float32), e)], 0.0).trigger
    assert not O.zen_auto_trigger([], 0.0).trigger


# ---------------------------------------------------------------- schedule

def _oracles(shapes, ratio, seed, R, S):
    rng = np.random.default_rng(seed)
    out = []
    for n, m in shapes:
        master = (0.02 * rng.standard_normal((n, m))).astype(np.float32)
        W = O.bf16_round(master)
        out.append(O.MatrixOracle(master, W, ratio, 1e-3, 0.9, 0.999, 1e-8, 0.0, R, S))
    return out


def _grads(shapes, T, seed):
    rng = np.random.default_rng(seed)
    res = []
    for _ in range(T):
        step = []
        for n, m in shapes:
            s = np.exp(1.5 * rng.standard_normal(m))
            step.append(bf16(rng.standard_normal((n, m)) * s))
        res.append(step)
    return res


def test_paper_example_point_one_reaches_point_five_in_five_steps():
    """Sensitivity of Hyperparameters: a low-importance gradient at 0.1 per
    step grows to 0.5 in five steps.  One selected channel of norm 1 (four
    rows of 0.5) and nine channels of norm ~0.1 (four rows of bf16(0.05))
    pointing the same way every step; with tau = 0.5 the hand-over fires at
    step 5, then again five steps later."""
    n, m = 4, 10
    G = np.full((n, m), 0.05, np.float32)
    G[:, 0] = 0.5
    Gb = bf16(G)
    master = np.zeros((n, m), np.float32)
    orc = O.MatrixOracle(master, O.bf16_round(master), 0.1, 1e-3, 0.9, 0.999, 1e-8, 0.0, 100, 8)
    za = O.ZenAutoOracle([orc], R=100, S_max=8, tau=0.5)
    ends = []
    for t in range(1, 13):
        r = za.step([Gb])
        if t == 1:
            assert list(orc.sel.sel) == [0]
        if r["interval_end"]:
            ends.append(t)
            # the hand-over is the mean of the interval: the gradient itself, up
            # to the one rounding of the 1/5 scale
            D = r["unpacked"][0]
            assert np.allclose(D[:, 1:], O.widen(Gb)[:, 1:], rtol=1e-6, atol=0)
            assert np.all(D[:, 0] == 0)
        norm = r["totals"].sum_acc / r["totals"].u
        assert abs(norm - r["step_in_interval"] * math.sqrt(4) * float(O.widen(Gb)[0, 1])) < 1e-6
    assert ends == [5, 10]
    za8 = O.ZenAutoOracle(_oracles([(n, m)], 0.1, 0, 100, 8), R=100, S_max=8, tau=math.inf)
    assert [t for t in range(1, 13) if za8.step([Gb])["interval_end"]] == [8]


@pytest.mark.parametrize("R,S", [(4, 4), (8, 4), (1, 4), (6, 3), (2, 2)])
def test_infinite_tau_is_the_fixed_schedule(R, S):
    """Holds when R is a multiple of S (then the fixed schedule's t mod S grid
    restarts at every refresh)."""
    shapes = [(9, 70), (16, 33)]
    T = 10
    grads = _grads(shapes, T, 5)
    fixed = _oracles(shapes, 0.2, 6, R, S)
    auto = _oracles(shapes, 0.2, 6, R, S)
    za = O.ZenAutoOracle(auto, R, S, math.inf)
    for t in range(1, T + 1):
        r = za.step(grads[t - 1])
        outs = [o.step(G) for o, G in zip(fixed, grads[t - 1])]
        kind = O.schedule(t, R, S)
        assert (r["refresh"], r["step_in_interval"], r["interval_end"]) == (
            kind.refresh, kind.step_in_interval, kind.interval_end)
        for a, b, of in zip(auto, fixed, outs):
            for x, y in ((a.P, b.P), (a.M, b.M), (a.V, b.V), (a.A, b.A), (a.W, b.W)):
                assert np.array_equal(x.view(np.uint32 if x.dtype == np.float32 else np.uint16),
                                      y.view(np.uint32 if y.dtype == np.float32 else np.uint16))
        if kind.interval_end:
            for D, of in zip(r["unpacked"], outs):
                assert np.array_equal(D.view(np.uint32), of["unpacked"].view(np.uint32))


def test_zero_tau_hands_over_every_step():
    shapes = [(5, 40)]
    grads = _grads(shapes, 7, 8)
    za = O.ZenAutoOracle(_oracles(shapes, 0.1, 9, 3, 4), 3, 4, 0.0)
    for t in range(1, 8):
        r = za.step(grads[t - 1])
        kind = O.schedule(t, 3, 1)
        assert (r["refresh"], r["step_in_interval"], r["interval_end"]) == (
            kind.refresh, kind.step_in_interval, kind.interval_end)
        assert r["totals"].trigger


@pytest.mark.parametrize("tau", [0.05, 0.1, 0.2, 0.4])
def test_schedule_invariants(tau):
    shapes = [(8, 50), (12, 21)]
    R, S = 5, 4
    T = 16
    grads = _grads(shapes, T, 10)
    za = O.ZenAutoOracle(_oracles(shapes, 0.1, 11, R, S), R, S, tau)
    prev_end = True
    lengths = []
    for t in range(1, T + 1):
        r = za.step(grads[t - 1])
        L = r["step_in_interval"]
        assert L == (1 if (prev_end or r["refresh"]) else lengths[-1] + 1)
        assert 1 <= L <= S
        want_end = r["totals"].trigger or L == S or (t % R == 0)
        assert r["interval_end"] == want_end
        # the totals are the plain sums of the per-matrix statistics
        tot = r["totals"]
        assert tot.k == sum(len(a) for a, _ in r["stats"])
        assert math.isclose(tot.sum_acc, sum(np.sqrt(b.astype(np.float64)).sum()
                                             for _, b in r["stats"]), rel_tol=1e-12)
        prev_end = r["interval_end"]
        lengths.append(L)
