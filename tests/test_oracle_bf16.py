"""Pins the oracle's bf16 <-> fp32 conversions against torch's CPU casts
(an independent library implementation of IEEE round-to-nearest-even)."""
import numpy as np
import pytest
import torch

from oracle import bf16_round, widen


def torch_round(x):
    return torch.from_numpy(np.asarray(x, np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)


def torch_widen(bits):
    return torch.from_numpy(np.asarray(bits, np.uint16).view(np.int16)).view(torch.bfloat16).float().numpy()


def _finite(u32):
    x = np.asarray(u32, dtype=np.uint32).view(np.float32)
    return x[np.isfinite(x) | np.isinf(x)]


def test_widen_all_patterns():
    bits = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    a = widen(bits)
    b = torch_widen(bits)
    nan = np.isnan(b)
    assert np.array_equal(a[~nan].view(np.uint32), b[~nan].view(np.uint32))
    assert np.isnan(a[nan]).all()


def test_round_ties_and_near_ties():
    hi = np.arange(0, 1 << 16, 7, dtype=np.uint32) << 16
    lows = np.array([0x0000, 0x0001, 0x7FFF, 0x8000, 0x8001, 0xFFFF], dtype=np.uint32)
    u = (hi[:, None] | lows[None, :]).ravel()
    x = _finite(u)
    assert np.array_equal(bf16_round(x), torch_round(x))


def test_round_random_patterns():
    rng = np.random.default_rng(7)
    x = _finite(rng.integers(0, 1 << 32, size=200_000, dtype=np.uint64).astype(np.uint32))
    assert np.array_equal(bf16_round(x), torch_round(x))


@pytest.mark.parametrize("u", [0x7F7FFFFF, 0x7F7F8000, 0x7F7F7FFF, 0x00000001, 0x00008000,
                               0x00018000, 0x807FFFFF, 0x80000000, 0x7F800000, 0xFF800000])
def test_round_edges(u):
    x = np.array([u], dtype=np.uint32).view(np.float32)
    assert np.array_equal(bf16_round(x), torch_round(x))


def test_round_nan_stays_nan():
    x = np.array([0x7FC00001, 0xFFFFFFFF, 0x7F800001], dtype=np.uint32).view(np.float32)
    assert np.isnan(widen(bf16_round(x))).all()
