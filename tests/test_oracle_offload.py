"""Pins of the oracle's offloaded-optimizer functions: the state swap at a
refresh against a full-state store (Zero-stall Pipeline, "Swapping out/in")
and the deferred update of the unselected columns with the interval's mean
gradient (Asynchronous Offloading Workflow; Convergence Analysis).

* swap_states: a hand-built leave / stay / enter example; the full optimizer
  state (store with the selected columns replaced by their compact states)
  is unchanged by any swap, bit for bit; with a store of (widened W, 0, 0)
  the compact states equal the pinned remap's.
* deferred_adam: equal, bit for bit, to the pinned adam_selected applied to
  the unselected columns when the buffer holds one widened gradient and the
  scale is 1; a dyadic 4-step sum with scale 1/4 is the exact mean; the
  first step from zero moments has the closed form; torch.optim.Adam (CPU,
  fp32) fed with the interval means agrees within 2e-6; selected columns of
  the store are untouched.
* OffloadOracle: ratio 0 is torch's Adam stepping once per interval on the
  mean gradient (the delayed-coordinate rule); ratio 1 is dense Adam every
  step; the full state is conserved across refreshes.
"""
import numpy as np
import pytest
import torch

import oracle as O

HP = dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.0)


def bf16(x):
    return O.bf16_round(np.asarray(x, dtype=np.float32))


def full_state(sel, P, M, V, store):
    """Every column's (p, m, v): compact states for selected columns, the
    store for the others."""
    out = [np.array(x, copy=True) for x in store]
    if sel is not None:
        for r, j in enumerate(sel.sel.tolist()):
            for dst, src in zip(out, (P, M, V)):
                dst[:, j] = src[:, r]
    return out


def sel_of(cols, m):
    s = np.zeros(m, np.float32)
    s[list(cols)] = 1.0
    return O.select_topk(s, len(cols))


# ---------------------------------------------------------------- swap

def test_swap_leave_stay_enter_example():
    n, m = 3, 5
    # store column j holds (100 + j, 200 + j, 300 + j); compact slot r of the
    # previous selection [1, 3] holds (10 + r, 20 + r, 30 + r)
    store = tuple(np.tile((base + np.arange(m)).astype(np.float32), (n, 1))
                  for base in (100, 200, 300))
    prev, new = sel_of([1, 3], m), sel_of([3, 4], m)
    P, M, V = (np.tile((base + np.arange(2)).astype(np.float32), (n, 1)) for base in (10, 20, 30))
    P2, M2, V2, (SP, SM, SV) = O.swap_states(prev, new, P, M, V, store)
    # column 3 stays (old slot 1 -> new slot 0); column 4 enters (new slot 1)
    assert np.all(P2[:, 0] == 11) and np.all(M2[:, 0] == 21) and np.all(V2[:, 0] == 31)
    assert np.all(P2[:, 1] == 104) and np.all(M2[:, 1] == 204) and np.all(V2[:, 1] == 304)
    # column 1 leaves: its compact states (old slot 0) go back to the store
    assert np.all(SP[:, 1] == 10) and np.all(SM[:, 1] == 20) and np.all(SV[:, 1] == 30)
    for j in (0, 2, 3, 4):
        assert np.all(SP[:, j] == 100 + j) and np.all(SM[:, j] == 200 + j)


@pytest.mark.parametrize("seed", range(5))
def test_swap_conserves_the_full_state(seed):
    rng = np.random.default_rng(seed)
    n, m = 6, 70
    store = tuple(rng.standard_normal((n, m)).astype(np.float32) for _ in range(3))
    prev = O.select_topk(rng.standard_normal(m).astype(np.float32), int(rng.integers(0, m + 1)))
    P, M, V = (rng.standard_normal((n, prev.k)).astype(np.float32) for _ in range(3))
    before = full_state(prev, P, M, V, store)
    new = O.select_topk(rng.standard_normal(m).astype(np.float32), int(rng.integers(0, m + 1)))
    P2, M2, V2, store2 = O.swap_states(prev, new, P, M, V, store)
    after = full_state(new, P2, M2, V2, store2)
    for a, b in zip(before, after):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


def test_swap_from_weight_store_equals_remap():
    rng = np.random.default_rng(7)
    n, m = 5, 40
    W = bf16(rng.standard_normal((n, m)) * 0.02)
    prev = O.select_topk(rng.standard_normal(m).astype(np.float32), 8)
    new = O.select_topk(rng.standard_normal(m).astype(np.float32), 8)
    P, M, V = (rng.standard_normal((n, 8)).astype(np.float32) for _ in range(3))
    store = (O.widen(W), np.zeros((n, m), np.float32), np.zeros((n, m), np.float32))
    got = O.swap_states(prev, new, P, M, V, store)[:3]
    want = O.remap(prev, new, P, M, V, W)
    for a, b in zip(got, want):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


def test_swap_first_selection_reads_everything_from_the_store():
    rng = np.random.default_rng(8)
    n, m = 4, 12
    store = tuple(rng.standard_normal((n, m)).astype(np.float32) for _ in range(3))
    new = sel_of([2, 5, 11], m)
    P2, M2, V2, store2 = O.swap_states(None, new, None, None, None, store)
    for got, s in zip((P2, M2, V2), store):
        assert np.array_equal(got, s[:, [2, 5, 11]])
    for a, b in zip(store, store2):
        assert np.array_equal(a, b)


# ---------------------------------------------------------------- deferred update

def test_deferred_equals_selected_adam_on_the_complement():
    rng = np.random.default_rng(1)
    n, m = 9, 31
    G = bf16(rng.standard_normal((n, m)) * np.exp(rng.standard_normal(m)))
    sel = O.select_topk(rng.standard_normal(m).astype(np.float32), 6)
    store = (rng.standard_normal((n, m)).astype(np.float32) * 0.02,
             rng.standard_normal((n, m)).astype(np.float32) * 1e-3,
             np.abs(rng.standard_normal((n, m))).astype(np.float32) * 1e-6)
    c = O.AdamConsts.at_step(**HP, t=3)
    A = O.widen(G[:, sel.unsel.astype(np.int64)])
    (SP, SM, SV), wun = O.deferred_adam(A, sel.unsel, 1.0, store, c)
    cols = sel.unsel.astype(np.int64)
    P1, M1, V1, w1 = O.adam_selected(G, sel.unsel, store[0][:, cols], store[1][:, cols],
                                     store[2][:, cols], c)
    for a, b in ((SP[:, cols], P1), (SM[:, cols], M1), (SV[:, cols], V1), (wun, w1)):
        assert np.array_equal(np.ascontiguousarray(a).view(np.uint8),
                              np.ascontiguousarray(b).view(np.uint8))
    scols = sel.sel.astype(np.int64)
    for a, b in zip((SP, SM, SV), store):
        assert np.array_equal(a[:, scols], b[:, scols])


def test_deferred_mean_of_dyadic_sum_is_exact_and_first_step_closed_form():
    rng = np.random.default_rng(2)
    n, u, S = 7, 11, 4
    ints = rng.integers(-64, 65, size=(S, n, u))
    ints[0, 0, 0] = 8  # at least one nonzero mean
    A = np.zeros((n, u), np.float32)
    for s in range(S):
        A = A + (ints[s] * 0.125).astype(np.float32)
    mean = ints.sum(0) * 0.125 / S
    z = np.zeros((n, u), np.float32)
    p0 = np.full((n, u), 0.5, np.float32)
    c = O.AdamConsts.at_step(**HP, t=1)
    (SP, SM, SV), _ = O.deferred_adam(A, np.arange(u), 0.25, (p0, z, z), c)
    # first step from zero moments: m' = (1-b1) g, v' = (1-b2) g^2,
    # p' = p0 - lr g / (|g| + eps) in reals
    assert np.all(np.abs(SM - 0.1 * mean) <= 2 * 2 ** -23 * np.abs(0.1 * mean))
    assert np.all(np.abs(SV - 1e-3 * mean ** 2) <= 4 * 2 ** -23 * 1e-3 * mean ** 2)
    want = 0.5 - 1e-3 * mean / (np.abs(mean) + 1e-8)
    assert np.all(np.abs(SP - want) <= 4 * 2 ** -24)


def test_deferred_matches_torch_adam_on_interval_means():
    rng = np.random.default_rng(3)
    n, m, S, intervals = 16, 12, 4, 3
    master = (rng.standard_normal((n, m)) * 0.02).astype(np.float32)
    p = torch.nn.Parameter(torch.from_numpy(master.copy()))
    opt = torch.optim.Adam([p], lr=1e-3, betas=(0.9, 0.999), eps=1e-8, foreach=False)
    orc = O.OffloadOracle(master, bf16(master), 0.0, 1e-3, 0.9, 0.999, 1e-8, 0.0, R=S, S=S)
    for _ in range(intervals):
        acc = np.zeros((n, m), np.float32)
        for _ in range(S):
            G = bf16(rng.standard_normal((n, m)) * np.exp(rng.standard_normal(m)))
            acc = (acc + O.widen(G)).astype(np.float32)
            out = orc.step(G)
        assert out["kind"].interval_end
        p.grad = torch.from_numpy((acc * np.float32(0.25)).astype(np.float32))
        opt.step()
    tp = p.detach().numpy()
    st = opt.state[p]
    assert np.all(np.abs(orc.store[0] - tp) <= 2e-6 * np.abs(tp) + 1e-9)
    assert np.all(np.abs(orc.store[2] - st["exp_avg_sq"].numpy())
                  <= 2e-6 * st["exp_avg_sq"].numpy())
    assert orc.th == intervals
    assert np.array_equal(orc.W, bf16(orc.store[0]))


def test_offload_ratio_one_is_dense_adam():
    rng = np.random.default_rng(4)
    n, m, T = 10, 16, 7
    master = (rng.standard_normal((n, m)) * 0.02).astype(np.float32)
    orc = O.OffloadOracle(master, bf16(master), 1.0, 1e-5, 0.9, 0.999, 1e-8, 0.0, R=3, S=2)
    p = torch.nn.Parameter(torch.from_numpy(master.copy()))
    opt = torch.optim.Adam([p], lr=1e-5, betas=(0.9, 0.999), eps=1e-8, foreach=False)
    for _ in range(T):
        G = bf16(rng.standard_normal((n, m)) * np.exp(rng.standard_normal(m)))
        orc.step(G)
        p.grad = torch.from_numpy(O.widen(G).copy())
        opt.step()
    tp = p.detach().numpy()
    assert np.all(np.abs(orc.P - tp) <= 2e-6 * np.abs(tp) + 1e-10)
    # intervals start at t = 1, 3, 4 (refresh), 5, 7: hand-overs at t = 2, 3, 4, 6
    assert [t for t in range(1, T + 1) if O.schedule(t, 3, 2).interval_end] == [2, 3, 4, 6]
    assert orc.th == 4
    assert np.array_equal(orc.W, bf16(orc.P))


def test_offload_conserves_state_through_refreshes():
    """Across refreshes with changing selections, every column's state
    evolves only through the two updates: a column's (p, m, v) in the full
    state after step t equals what the previous full state gives by one
    selected-Adam step (selected columns) or is unchanged (unselected ones,
    between hand-overs)."""
    rng = np.random.default_rng(5)
    n, m = 6, 40
    master = (rng.standard_normal((n, m)) * 0.02).astype(np.float32)
    orc = O.OffloadOracle(master, bf16(master), 0.25, 1e-3, 0.9, 0.999, 1e-8, 0.0, R=1, S=3)
    prev_full = None
    for t in range(1, 7):
        G = bf16(rng.standard_normal((n, m)) * np.exp(2 * rng.standard_normal(m)))
        kind = O.schedule(t, 1, 3)
        assert kind.interval_end  # R = 1: every step ends its interval
        before = full_state(orc.sel, orc.P, orc.M, orc.V, orc.store)
        orc.step(G)
        after = full_state(orc.sel, orc.P, orc.M, orc.V, orc.store)
        # selected columns: one Adam step at global t from the state before
        c = O.AdamConsts.at_step(1e-3, 0.9, 0.999, 1e-8, 0.0, t)
        cols = orc.sel.sel.astype(np.int64)
        P1, M1, V1, _ = O.adam_selected(G, orc.sel.sel, before[0][:, cols], before[1][:, cols],
                                        before[2][:, cols], c)
        for a, b in zip((P1, M1, V1), after):
            assert np.array_equal(a, b[:, cols])
        # unselected columns: one deferred step (host step t) on g = G
        ch = O.AdamConsts.at_step(1e-3, 0.9, 0.999, 1e-8, 0.0, orc.th)
        ucols = orc.sel.unsel.astype(np.int64)
        P1, M1, V1, _ = O.adam_selected(G, orc.sel.unsel, before[0][:, ucols],
                                        before[1][:, ucols], before[2][:, ucols], ch)
        for a, b in zip((P1, M1, V1), after):
            assert np.array_equal(a, b[:, ucols])
        prev_full = after
    assert prev_full is not None


def test_zen_auto_drives_the_deferred_update():
    """ZenAutoOracle over OffloadOracles: with tau = inf it is the fixed
    schedule with S = S_max (R a multiple of S_max) bit for bit; with tau = 0
    every step hands over, i.e. the deferred update runs after every step."""
    rng = np.random.default_rng(9)
    shapes = [(6, 40), (9, 17)]
    masters = [(rng.standard_normal(s) * 0.02).astype(np.float32) for s in shapes]
    grads = [[bf16(rng.standard_normal(s) * np.exp(rng.standard_normal(s[1]))) for s in shapes]
             for _ in range(9)]

    def make(R, S):
        return [O.OffloadOracle(mw, bf16(mw), 0.25, 1e-3, 0.9, 0.999, 1e-8, 0.0, R, S)
                for mw in masters]

    za = O.ZenAutoOracle(make(6, 3), R=6, S_max=3, tau=float("inf"))
    fixed = make(6, 3)
    for step in grads:
        r = za.step(step)
        outs = [o.step(G) for o, G in zip(fixed, step)]
        assert r["interval_end"] == outs[0]["kind"].interval_end
    for a, b in zip(za.orcs, fixed):
        assert a.th == b.th == 3
        for x, y in zip(a.store, b.store):
            assert np.array_equal(x.view(np.uint32), y.view(np.uint32))
        assert np.array_equal(a.W, b.W)
    za0 = O.ZenAutoOracle(make(6, 3), R=6, S_max=3, tau=0.0)
    for step in grads:
        assert za0.step(step)["interval_end"]
    assert all(o.th == len(grads) for o in za0.orcs)


def test_warmup_steps_are_not_stale():
    """During the warm-up every step hands over (intervals of one step), so
    with nothing selected the offloaded optimizer is torch's Adam stepping on
    every gradient (no accumulation, no staleness)."""
    rng = np.random.default_rng(11)
    n, m, T = 12, 10, 6
    master = (rng.standard_normal((n, m)) * 0.02).astype(np.float32)
    orc = O.OffloadOracle(master, bf16(master), 0.0, 1e-3, 0.9, 0.999, 1e-8, 0.0, R=4, S=4,
                          warmup=T)
    p = torch.nn.Parameter(torch.from_numpy(master.copy()))
    opt = torch.optim.Adam([p], lr=1e-3, betas=(0.9, 0.999), eps=1e-8, foreach=False)
    for _ in range(T):
        G = bf16(rng.standard_normal((n, m)) * np.exp(rng.standard_normal(m)))
        assert orc.step(G)["kind"].interval_end
        p.grad = torch.from_numpy(O.widen(G).copy())
        opt.step()
    tp = p.detach().numpy()
    assert orc.th == T
    assert np.all(np.abs(orc.store[0] - tp) <= 2e-6 * np.abs(tp) + 1e-9)
