"""Pins the oracle's pack/accumulate and unpack: the unpack(pack) identity
against torch's independent bf16 widening, exact dyadic S-step sums, the
overwrite rule at interval start, and the paper's I/O-model figure."""
import numpy as np
import pytest
import torch

from oracle import MatrixOracle, bf16_round, pack_accumulate, select_topk, unpack
from tests._golden import read_keyvals


def torch_widen(bits):
    return torch.from_numpy(np.asarray(bits, np.uint16).view(np.int16)).view(torch.bfloat16).float().numpy()


def test_unpack_of_pack_is_identity_on_unselected_columns():
    rng = np.random.default_rng(0)
    n, m = 33, 130
    G = bf16_round((rng.standard_normal((n, m)) * 3).astype(np.float32))
    G[0, :] = 0x8000  # -0.0 must survive bitwise
    sel = select_topk(rng.random(m).astype(np.float32), 13)
    A = pack_accumulate(G, sel.unsel, None, 1)
    assert A.shape == (n, m - 13)
    D = unpack(A, sel, 1.0)
    ref = torch_widen(G)
    assert np.array_equal(D[:, sel.unsel].view(np.uint32), ref[:, sel.unsel].view(np.uint32))
    assert np.all(D[:, sel.sel].view(np.uint32) == 0)  # +0.0


def test_interval_start_overwrites():
    G = np.array([[0x3F80, 0x8000]], np.uint16)  # 1.0, -0.0
    sel = select_topk(np.array([0.0, 0.0], np.float32), 0)
    junk = np.array([[np.nan, 5.0]], np.float32)
    A = pack_accumulate(G, sel.unsel, junk, 1)
    assert A.view(np.uint32).tolist() == [[0x3F800000, 0x80000000]]


@pytest.mark.parametrize("S", [2, 4, 8])
def test_dyadic_sums_are_exact(S):
    rng = np.random.default_rng(S)
    n, m = 9, 70
    ints = rng.integers(-255, 256, size=(S, n, m))
    sel = select_topk(rng.random(m).astype(np.float32), 7)
    A = None
    for s in range(S):
        G = bf16_round((ints[s] * 0.125).astype(np.float32))
        A = pack_accumulate(G, sel.unsel, A, s + 1)
    want = ints.sum(axis=0)[:, sel.unsel] * 0.125
    assert np.array_equal(A, want.astype(np.float32))
    D = unpack(A, sel, 1.0 / S)
    assert np.array_equal(D[:, sel.unsel], (want / S).astype(np.float32))


def test_io_model_volume_matches_paper():
    """Per interval of S steps the unselected part moves (m - k) columns each
    step and once more when the interval is handed over."""
    g = read_keyvals("paper_numbers.txt")
    S, ratio = g["io_S"], g["io_ratio"]
    n, m = 2, 40
    rng = np.random.default_rng(1)
    W = bf16_round((rng.standard_normal((n, m)) * 0.02).astype(np.float32))
    orc = MatrixOracle(W.astype(np.float32), W, ratio, 1e-5, 0.9, 0.999, 1e-8, 0.0, R=S, S=S)
    moved = 0
    for t in range(S):
        G = bf16_round(rng.standard_normal((n, m)).astype(np.float32))
        out = orc.step(G)
        moved += orc.A.shape[1]
        if "unpacked" in out:
            moved += orc.sel.unsel.size
    assert moved / (S * m) == pytest.approx(g["io_per_iteration"], abs=1e-12)
