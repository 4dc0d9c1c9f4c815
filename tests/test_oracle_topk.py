"""Pins the oracle's top-k column selection against brute force over all
subsets, the selection invariants, and the k table."""
import itertools

import numpy as np
import pytest

from oracle import k_from_ratio, select_topk, slots_of
from tests._golden import read_table
from workloads import score_vector


def brute_force(s, k):
    """First subset (in lexicographic order of sorted indices) whose every
    member scores at least as high as every non-member.  Lexicographic order
    makes the lowest indices win among tied scores."""
    m = len(s)
    for combo in itertools.combinations(range(m), k):
        chosen = set(combo)
        lo = min((s[j] for j in chosen), default=float("inf"))
        hi = max((s[j] for j in range(m) if j not in chosen), default=float("-inf"))
        if lo >= hi:
            return list(combo)
    raise AssertionError("no valid subset")


def check_mask_prefix(sel, m):
    chosen = set(sel.sel.tolist())
    words = (m + 63) // 64
    assert sel.mask.shape == (words,) and sel.prefix.shape == (words,)
    for w in range(words):
        for b in range(64):
            j = 64 * w + b
            bit = (int(sel.mask[w]) >> b) & 1
            assert bit == (1 if j in chosen else 0)
        assert sel.prefix[w] == sum(1 for j in chosen if j < 64 * w)


@pytest.mark.parametrize("m", [1, 2, 3, 4, 5, 6])
def test_brute_force_all_tie_patterns(m):
    for vals in itertools.product([0.0, 1.0, 2.0], repeat=m):
        s = np.array(vals, dtype=np.float32)
        for k in range(m + 1):
            got = select_topk(s, k)
            assert got.sel.tolist() == brute_force(list(vals), k), (vals, k)
            assert got.unsel.tolist() == sorted(set(range(m)) - set(got.sel.tolist()))


@pytest.mark.parametrize("m", [3, 5])
def test_signed_zero_ties_with_positive_zero(m):
    for vals in itertools.product([-0.0, 0.0, 1.0], repeat=m):
        s = np.array(vals, dtype=np.float32)
        for k in range(m + 1):
            assert select_topk(s, k).sel.tolist() == brute_force(list(vals), k)


@pytest.mark.parametrize("kind", ["lognormal", "wide", "ties", "few-distinct", "constant", "zeros"])
@pytest.mark.parametrize("m", [7, 64, 65, 1000, 4096])
def test_invariants(kind, m):
    s = score_vector(m, seed=m, kind=kind).numpy()
    for k in sorted({0, 1, m // 3, k_from_ratio(0.1, m), m - 1, m}):
        sel = select_topk(s, k)
        a, b = sel.sel.tolist(), sel.unsel.tolist()
        assert len(a) == k and len(b) == m - k
        assert sorted(a + b) == list(range(m))
        assert a == sorted(a) and b == sorted(b)
        if 0 < k < m:
            t = min(s[a])
            assert t >= max(s[b])
            tied_sel = [j for j in a if s[j] == t]
            tied_uns = [j for j in b if s[j] == t]
            if tied_uns:
                assert max(tied_sel) < min(tied_uns)
        check_mask_prefix(sel, m)


def test_slots():
    sel = select_topk(np.array([5, 1, 4, 2, 3], np.float32), 2)
    assert sel.sel.tolist() == [0, 2]
    assert slots_of(sel.sel, 5).tolist() == [0, -1, 1, -1, -1]
    assert slots_of(sel.unsel, 5).tolist() == [-1, 0, -1, 1, 2]


def test_k_table():
    rows = read_table("k_table.txt")
    ratios = [0.01, 0.05, 0.10, 0.25]
    for row in rows:
        m = int(row[0])
        for r, want in zip(ratios, row[1:]):
            assert k_from_ratio(r, m) == int(want), (m, r)


def test_k_edges():
    assert k_from_ratio(0.0, 10) == 0 and k_from_ratio(1.0, 10) == 10
    assert k_from_ratio(0.25, 2) == 1   # 0.5 rounds up
    assert k_from_ratio(0.5, 0) == 0
    for bad in (-0.1, 1.1, float("nan")):
        with pytest.raises(ValueError):
            k_from_ratio(bad, 10)
