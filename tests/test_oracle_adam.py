"""Pins the oracle's selective Adam against closed forms and against
torch.optim.Adam / AdamW on the CPU (an independent implementation)."""
import numpy as np
import pytest
import torch

from oracle import AdamConsts, adam_selected, bf16_round, remap, select_topk, widen

HP = dict(lr=1e-5, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.0)


def ulp32(x):
    x = np.abs(np.asarray(x, np.float32))
    return np.spacing(x).astype(np.float64)


def grads(rng, n, m, scale=1.0):
    g = (rng.standard_normal((n, m)) * scale).astype(np.float32)
    return bf16_round(g)


def test_first_step_closed_form():
    rng = np.random.default_rng(0)
    n, m = 64, 48
    G = grads(rng, n, m, scale=np.exp(rng.standard_normal(m) * 1.5))
    sel = np.arange(m, dtype=np.int32)
    P = (rng.standard_normal((n, m)) * 0.02).astype(np.float32)
    Z = np.zeros((n, m), np.float32)
    c = AdamConsts.at_step(**HP, t=1)
    P1, M1, V1, W = adam_selected(G, sel, P, Z, Z, c)
    g = widen(G).astype(np.float64)
    # m' = (1-b1) g and v' = (1-b2) g^2, each one or two fp32 roundings away.
    assert np.all(np.abs(M1 - 0.1 * g) <= 1.0 * ulp32(M1) + 1e-12 * np.abs(g))
    assert np.all(np.abs(V1 - 0.001 * g * g) <= 2.0 * ulp32(V1))
    # Bias correction makes the first step exactly p - lr * g / (|g| + eps) in reals.
    exact = P.astype(np.float64) - 1e-5 * g / (np.abs(g) + 1e-8)
    assert np.all(np.abs(P1 - exact) <= ulp32(P1) + 1e-6 * 1e-5)
    assert np.array_equal(W, bf16_round(P1))


def test_constant_gradient_closed_form():
    rng = np.random.default_rng(1)
    n, m, T = 16, 40, 12
    G = grads(rng, n, m, scale=np.exp(rng.standard_normal(m)))
    sel = np.arange(m, dtype=np.int32)
    P0 = (rng.standard_normal((n, m)) * 0.02).astype(np.float32)
    P, M, V = P0.copy(), np.zeros((n, m), np.float32), np.zeros((n, m), np.float32)
    for t in range(1, T + 1):
        P, M, V, _ = adam_selected(G, sel, P, M, V, AdamConsts.at_step(**HP, t=t))
    g = widen(G).astype(np.float64)
    # With a constant g, m_hat = g and v_hat = g^2 at every step (in reals).
    exact = P0.astype(np.float64) - T * 1e-5 * g / (np.abs(g) + 1e-8)
    assert np.all(np.abs(P - exact) <= T * ulp32(P0) + 1e-5 * T * 1e-5)
    assert np.allclose(M, (1 - 0.9 ** T) * g, rtol=1e-5, atol=0)
    assert np.allclose(V, (1 - 0.999 ** T) * g * g, rtol=1e-5, atol=0)


def test_decoupled_weight_decay_closed_form():
    n, m = 4, 8
    P = np.linspace(-1, 1, n * m, dtype=np.float32).reshape(n, m)
    G = np.zeros((n, m), np.uint16)
    Z = np.zeros((n, m), np.float32)
    hp = dict(HP, weight_decay=0.1)
    P1, M1, V1, _ = adam_selected(G, np.arange(m, dtype=np.int32), P, Z, Z,
                                  AdamConsts.at_step(**hp, t=3))
    assert np.all(M1 == 0) and np.all(V1 == 0)
    assert np.all(np.abs(P1 - P.astype(np.float64) * (1 - 1e-6)) <= ulp32(P1))


@pytest.mark.parametrize("wd", [0.0, 0.01])
def test_matches_torch_adam_when_everything_is_selected(wd):
    rng = np.random.default_rng(2)
    n, m, T = 32, 24, 6
    P0 = (rng.standard_normal((n, m)) * 0.02).astype(np.float32)
    p = torch.nn.Parameter(torch.from_numpy(P0.copy()))
    opt_cls = torch.optim.AdamW if wd else torch.optim.Adam
    opt = opt_cls([p], lr=1e-5, betas=(0.9, 0.999), eps=1e-8, weight_decay=wd, foreach=False)
    P, M, V = P0.copy(), np.zeros((n, m), np.float32), np.zeros((n, m), np.float32)
    sel = np.arange(m, dtype=np.int32)
    hp = dict(HP, weight_decay=wd)
    gmax = np.zeros((n, m))
    for t in range(1, T + 1):
        G = grads(rng, n, m, scale=np.exp(rng.standard_normal(m)))
        gmax = np.maximum(gmax, np.abs(widen(G)))
        p.grad = torch.from_numpy(widen(G).copy())
        opt.step()
        P, M, V, _ = adam_selected(G, sel, P, M, V, AdamConsts.at_step(**hp, t=t))
    st = opt.state[p]
    tp, tm, tv = p.detach().numpy(), st["exp_avg"].numpy(), st["exp_avg_sq"].numpy()
    assert np.all(np.abs(P - tp) <= 2e-6 * np.abs(tp) + 1e-6 * 1e-5)
    assert np.all(np.abs(V - tv) <= 2e-6 * np.abs(tv))
    # m can cancel; floor the tolerance at the size of the terms it sums.
    assert np.all(np.abs(M - tm) <= 2e-6 * np.abs(tm) + 2e-6 * 0.1 * gmax)


def test_only_selected_columns_are_touched():
    rng = np.random.default_rng(3)
    n, m = 8, 20
    G = grads(rng, n, m)
    s = np.arange(m, dtype=np.float32)[::-1].copy()
    sel = select_topk(s, 5)
    assert sel.sel.tolist() == [0, 1, 2, 3, 4]
    P = rng.standard_normal((n, 5)).astype(np.float32)
    Z = np.zeros((n, 5), np.float32)
    P1, _, _, _ = adam_selected(G, sel.sel, P, Z, Z, AdamConsts.at_step(**HP, t=1))
    P1b, _, _, _ = adam_selected(G[:, :5].copy(), np.arange(5, dtype=np.int32), P, Z, Z,
                                 AdamConsts.at_step(**HP, t=1))
    assert np.array_equal(P1, P1b)


def test_remap_moves_surviving_states_and_initialises_new_ones():
    n, m = 3, 10
    old = select_topk(np.array([9, 0, 8, 0, 7, 0, 0, 6, 0, 0], np.float32), 4)  # 0,2,4,7
    new = select_topk(np.array([0, 9, 8, 0, 0, 0, 0, 7, 6, 0], np.float32), 4)  # 1,2,7,8
    P = np.arange(n * 4, dtype=np.float32).reshape(n, 4) + 100
    M = -P
    V = P * 2
    W = bf16_round(np.arange(n * m, dtype=np.float32).reshape(n, m) * 0.5)
    P2, M2, V2 = remap(old, new, P, M, V, W)
    # columns 2 and 7 survive: old slots 1 and 3 -> new slots 1 and 2
    assert np.array_equal(P2[:, 1], P[:, 1]) and np.array_equal(P2[:, 2], P[:, 3])
    assert np.array_equal(M2[:, 2], M[:, 3]) and np.array_equal(V2[:, 1], V[:, 1])
    # columns 1 and 8 are new: p from the widened weight, zero moments
    assert np.array_equal(P2[:, 0], widen(W[:, 1])) and np.array_equal(P2[:, 3], widen(W[:, 8]))
    assert np.all(M2[:, [0, 3]] == 0) and np.all(V2[:, [0, 3]] == 0)
    master = np.full((n, m), 0.125, np.float32)
    P3, _, _ = remap(None, new, None, None, None, W, master)
    assert np.all(P3 == 0.125)


def test_eps_outside_the_square_root_for_tiny_gradients():
    # |g| comparable to eps separates g/(|g|+eps) from g/sqrt(g^2+eps) and
    # from g/sqrt(g^2+eps^2).
    n, m = 4, 6
    gv = np.array([1e-8, -3e-9, 2e-8, 5e-10, -1e-7, 4e-9], np.float32)
    G = bf16_round(np.tile(gv, (n, 1)))
    g = widen(G).astype(np.float64)
    P = np.zeros((n, m), np.float32)
    Z = np.zeros((n, m), np.float32)
    P1, _, _, _ = adam_selected(G, np.arange(m, dtype=np.int32), P, Z, Z, AdamConsts.at_step(**HP, t=1))
    exact = -1e-5 * g / (np.abs(g) + 1e-8)
    assert np.allclose(P1, exact, rtol=1e-5, atol=0)
    assert not np.allclose(P1, -1e-5 * g / np.sqrt(g * g + 1e-8), rtol=1e-2)
