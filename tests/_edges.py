"""Inputs and comparisons shared by the Adam edge-value tests (host and
device): seeded edge patterns for one selective step, and a bitwise
comparison under which NaN matches NaN whatever its payload."""
import numpy as np

import oracle as O
from workloads import derive_seed, edge_bf16, edge_f32, sprinkle_nonfinite


def same_nan_aware(got, want) -> bool:
    """Bitwise equal, except that NaN matches NaN whatever its payload."""
    got = np.ascontiguousarray(got, np.float32)
    want = np.ascontiguousarray(want, np.float32)
    if got.shape != want.shape:
        return False
    gn, wn = np.isnan(got), np.isnan(want)
    if not np.array_equal(gn, wn):
        return False
    return bool(np.array_equal(got[~gn].view(np.uint32), want[~wn].view(np.uint32)))


def first_mismatch(got, want):
    got = np.ascontiguousarray(got, np.float32)
    want = np.ascontiguousarray(want, np.float32)
    bad = ~((got.view(np.uint32) == want.view(np.uint32)) | (np.isnan(got) & np.isnan(want)))
    idx = np.argwhere(bad)
    if idx.size == 0:
        return None
    i = tuple(idx[0])
    return i, float(got[i]), float(want[i]), int(bad.sum())


def bf16_as_f32(bits):
    return O.widen(np.asarray(bits, np.uint16))


def inputs(n, m, ratio, seed, nonfinite):
    rng = np.random.default_rng(derive_seed("adam-edges", n, m, seed))
    k = O.k_from_ratio(ratio, m)
    sel = O.select_topk(rng.random(m).astype(np.float32), k)
    G = edge_bf16((n, m), derive_seed("g", n, m, seed))
    P = edge_f32((n, k), derive_seed("p", n, m, seed), "master")
    Mo = edge_f32((n, k), derive_seed("m", n, m, seed), "first")
    V = edge_f32((n, k), derive_seed("v", n, m, seed), "second")
    if nonfinite:
        Mo, V = sprinkle_nonfinite(Mo, V, derive_seed("nf", n, m, seed))
    W = edge_bf16((n, m), derive_seed("w", n, m, seed))
    A = edge_f32((n, m - k), derive_seed("a", n, m, seed), "sum")
    master = edge_f32((n, m), derive_seed("master", n, m, seed), "master")
    return G, sel, P, Mo, V, W, A, master
