"""The seeded generator: determinism, shapes, parameter totals, and the
column-spacing property checked with the oracle's scores."""
import numpy as np
import pytest
import torch

from oracle import colnorm, k_from_ratio, select_topk
from workloads import (WORKLOADS, derive_seed, get_workload, gradient, gradient_iid,
                       master_weights, space_all_pairs, space_boundary, step_scales)


def bits(t):
    return t.contiguous().view(torch.int16).numpy().view(np.uint16)


def test_parameter_totals():
    assert get_workload("linear-4096x4096").params == 16_777_216
    assert get_workload("llama2-7b-layer").params == 202_375_168
    assert get_workload("llama2-7b-full").params == 6_738_149_376
    assert get_workload("llama2-13b-full").params == 13_015_449_600
    assert get_workload("llama2-70b-10layers").params == 8_556_380_160
    assert len(get_workload("llama2-7b-full").matrices) == 226


def test_determinism():
    s = step_scales(get_workload("llama2-7b-layer"), 0, 2)
    a = gradient(64, 96, s[:96], seed=5)
    b = gradient(64, 96, s[:96], seed=5)
    c = gradient(64, 96, s[:96], seed=6)
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    assert not torch.equal(a.view(torch.int16), c.view(torch.int16))
    assert torch.equal(master_weights(8, 8, 3), master_weights(8, 8, 3))


def test_independent_draws():
    """gradient_iid: the same seed gives the same bits; each column's energy
    divided by s_j^2 varies from column to column (its own noise), where the
    shifted-copy generator gives the same ratio for every column up to bf16
    rounding; the mean of those ratios is about 1 (elements N(0, 1) * s_j)."""
    n, m = 512, 200
    sc = torch.exp(torch.randn(m, generator=torch.Generator().manual_seed(3),
                               dtype=torch.float64))
    a = gradient_iid(n, m, sc, seed=9)
    assert torch.equal(a.view(torch.int16), gradient_iid(n, m, sc, seed=9).view(torch.int16))
    assert not torch.equal(a.view(torch.int16), gradient_iid(n, m, sc, seed=10).view(torch.int16))
    s2 = sc.numpy() ** 2
    ratio_iid = colnorm(bits(a)).astype(np.float64) / s2 / n
    ratio_shift = colnorm(bits(gradient(n, m, sc, seed=9))).astype(np.float64) / s2 / n
    assert np.std(ratio_shift) < 2e-3                       # one noise energy for all
    assert 0.03 < np.std(ratio_iid) < 0.12                  # sqrt(2 / n) = 0.0625
    assert abs(np.mean(ratio_iid) - 1.0) < 0.03


def test_all_pairs_spacing_of_realised_scores():
    n, m = 1024, 1024
    s = space_all_pairs(torch.exp(1.5 * torch.randn(m, generator=torch.Generator().manual_seed(1),
                                                    dtype=torch.float64)))
    G = bits(gradient(n, m, s, seed=derive_seed("spacing")))
    sc = np.sort(colnorm(G).astype(np.float64))
    assert ((sc[1:] - sc[:-1]) / sc[:-1]).min() > 1e-3


def test_boundary_spacing_of_realised_scores():
    n, m = 2048, 4096
    k = k_from_ratio(0.1, m)
    wl = get_workload("llama2-7b-layer")
    s = step_scales(wl, 0, 1, k_boundary=k)
    G = bits(gradient(n, m, s, seed=derive_seed(wl.seed, 0, "grad", 1)))
    sc = colnorm(G).astype(np.float64)
    order = np.sort(sc)[::-1]
    assert (order[k - 1] - order[k]) / order[k] > 1e-3
    # the selection by realised scores is the selection by scales
    assert select_topk(sc.astype(np.float32), k).sel.tolist() == sorted(
        np.argsort(-s.numpy(), kind="stable")[:k].tolist())


def test_spacing_helpers_keep_order():
    s = torch.exp(torch.randn(500, generator=torch.Generator().manual_seed(2), dtype=torch.float64))
    a = space_all_pairs(s)
    assert torch.equal(torch.argsort(a), torch.argsort(s))
    b = space_boundary(s, 50)
    assert torch.equal(torch.argsort(b), torch.argsort(s))


def test_gradient_into_strided_view():
    buf = torch.zeros(7, 16, dtype=torch.bfloat16)
    view = buf[:, :13]
    s = torch.ones(13, dtype=torch.float64)
    gradient(7, 13, s, seed=1, out=view)
    assert torch.equal(view.view(torch.int16), gradient(7, 13, s, seed=1).view(torch.int16))
    assert torch.all(buf[:, 13:] == 0)


@pytest.mark.parametrize("name", sorted(WORKLOADS))
def test_workload_fields(name):
    wl = WORKLOADS[name]
    assert 0 < wl.ratio <= 1 and wl.refresh >= 1 and wl.accum >= 1 and wl.steps >= 1
    for mt in wl.matrices:
        assert mt.n > 0 and mt.m > 0
