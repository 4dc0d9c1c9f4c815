"""Pins the per-step composition of the oracle (MatrixOracle) at the two
degenerate selection ratios, where the method reduces to known routines:
ratio 1 -> plain Adam on the whole matrix (torch.optim.Adam on the CPU);
ratio 0 -> plain accumulation of every column (exact dyadic sums)."""
import numpy as np
import torch

from oracle import MatrixOracle, bf16_round, widen


def test_ratio_one_is_dense_adam_across_refreshes():
    rng = np.random.default_rng(0)
    n, m, T = 12, 20, 7
    master = (rng.standard_normal((n, m)) * 0.02).astype(np.float32)
    W = bf16_round(master)
    orc = MatrixOracle(master, W, 1.0, 1e-5, 0.9, 0.999, 1e-8, 0.0, R=3, S=2)
    p = torch.nn.Parameter(torch.from_numpy(master.copy()))
    opt = torch.optim.Adam([p], lr=1e-5, betas=(0.9, 0.999), eps=1e-8, foreach=False)
    for t in range(T):
        G = bf16_round((rng.standard_normal((n, m)) * np.exp(rng.standard_normal(m))).astype(np.float32))
        out = orc.step(G)
        p.grad = torch.from_numpy(widen(G).copy())
        opt.step()
        if "unpacked" in out:
            assert np.all(out["unpacked"].view(np.uint32) == 0)
    tp = p.detach().numpy()
    assert np.all(np.abs(orc.P - tp) <= 2e-6 * np.abs(tp) + 1e-10)
    assert np.array_equal(orc.W, bf16_round(orc.P))


def test_ratio_zero_accumulates_everything():
    rng = np.random.default_rng(1)
    n, m, S = 5, 9, 4
    W = np.zeros((n, m), np.uint16)
    orc = MatrixOracle(np.zeros((n, m), np.float32), W, 0.0, 1e-5, 0.9, 0.999, 1e-8, 0.0, R=S, S=S)
    total = np.zeros((n, m), np.int64)
    for t in range(S):
        ints = rng.integers(-100, 101, size=(n, m))
        total += ints
        out = orc.step(bf16_round((ints * 0.25).astype(np.float32)))
    assert np.array_equal(out["unpacked"], (total * 0.25 / S).astype(np.float32))
    assert np.all(orc.W == 0)
