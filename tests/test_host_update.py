"""The deferred host update of the unselected columns (zf_host_adam_unselected,
host code of libzf) against the oracle's deferred_adam: bit for bit, in both
layouts, on ragged shapes, padded strides, 1 and several threads, with and
without decoupled weight decay; host-side validation.  No GPU is involved:
the function takes host pointers only."""
import ctypes

import numpy as np
import pytest
import torch

import oracle as O

zf = pytest.importorskip("paper_2505_12242_amd")
from paper_2505_12242_amd import _lib  # noqa: E402


def _case(n, m, ratio, seed, wd=0.0, step=3):
    rng = np.random.default_rng(seed)
    k = O.k_from_ratio(ratio, m)
    sel = O.select_topk(rng.standard_normal(m).astype(np.float32), k)
    u = m - k
    A = (rng.standard_normal((n, u)) * np.exp(rng.standard_normal(u))).astype(np.float32)
    store = ((rng.standard_normal((n, m)) * 0.02).astype(np.float32),
             (rng.standard_normal((n, m)) * 1e-3).astype(np.float32),
             (np.abs(rng.standard_normal((n, m))) * 1e-6).astype(np.float32))
    hp = zf.AdamHparams(lr=1e-3, weight_decay=wd)
    c = O.AdamConsts.at_step(hp.lr, hp.beta1, hp.beta2, hp.eps, hp.weight_decay, step)
    return sel, A, store, hp, c


def _store_t(x, layout, pad):
    """Host tensor of logical [r, c] array x in `layout`, rows padded by pad."""
    x = x if layout == zf.ROW_MAJOR else np.ascontiguousarray(x.T)
    r, c = x.shape
    buf = torch.full((r, c + pad), float("nan"), dtype=torch.float32)
    buf[:, :c] = torch.from_numpy(x)
    return buf[:, :c]


def _logical(t, layout):
    a = t.numpy() if t.dtype != torch.bfloat16 else t.view(torch.int16).numpy().view(np.uint16)
    return a if layout == zf.ROW_MAJOR else np.ascontiguousarray(a.T)


@pytest.mark.parametrize("layout", [0, 1])
@pytest.mark.parametrize("n,m,ratio", [(1, 1, 0.0), (3, 7, 0.3), (64, 130, 0.1),
                                       (257, 33, 0.1), (40, 1000, 0.05), (17, 9, 1.0)])
@pytest.mark.parametrize("threads", [1, 5])
def test_host_update_matches_oracle(layout, n, m, ratio, threads):
    sel, A, store, hp, c = _case(n, m, ratio, seed=n * 1000 + m)
    want_store, want_w = O.deferred_adam(A, sel.unsel, 0.25, store, c)
    u = m - sel.k
    acc = _store_t(A, layout, 3)
    P, M, V = (_store_t(x, layout, 5) for x in store)
    wr, wc = (n, u) if layout == 0 else (u, n)
    wcols = torch.zeros(wr, wc + 2, dtype=torch.bfloat16)[:, :wc]
    unsel = torch.from_numpy(sel.unsel.astype(np.int32))
    zf.host_adam_unselected(acc, unsel, n, m, sel.k, 0.25, P, M, V, wcols, hp, step=3,
                            layout=layout, nthreads=threads)
    for got, want in zip((P, M, V), want_store):
        assert np.array_equal(_logical(got, layout).view(np.uint32), want.view(np.uint32))
    assert np.array_equal(_logical(wcols, layout), want_w)


def test_host_update_decay_and_threads_are_bit_identical():
    sel, A, store, hp, c = _case(128, 600, 0.1, seed=5, wd=0.05, step=7)
    want_store, want_w = O.deferred_adam(A, sel.unsel, 1.0 / 3.0, store, c)
    outs = []
    for threads in (1, 3, 16):
        P, M, V = (torch.from_numpy(x.copy()) for x in store)
        wcols = torch.zeros(128, 600 - sel.k, dtype=torch.bfloat16)
        zf.host_adam_unselected(torch.from_numpy(A), torch.from_numpy(sel.unsel.astype(np.int32)),
                                128, 600, sel.k, float(np.float32(1.0 / 3.0)), P, M, V, wcols,
                                hp, step=7, nthreads=threads)
        outs.append((P.numpy().tobytes(), M.numpy().tobytes(), V.numpy().tobytes(),
                     wcols.view(torch.int16).numpy().tobytes()))
        assert np.array_equal(P.numpy(), want_store[0])
        assert np.array_equal(wcols.view(torch.int16).numpy().view(np.uint16), want_w)
    assert outs[0] == outs[1] == outs[2]


def _raw(acc, ld_acc, unsel, n, m, k, layout, P, ld_state, W, ld_w, step=1, scale=1.0,
         threads=1):
    hp = _lib.ZfAdamHparams(1e-3, 0.9, 0.999, 1e-8, 0.0)
    return _lib.LIB.zf_host_adam_unselected(acc, ld_acc, unsel, n, m, k, layout, scale, P,
                                            P + 4 * ld_state * n if P else None,
                                            P + 8 * ld_state * n if P else None, ld_state, W,
                                            ld_w, ctypes.byref(hp), step, threads)


def test_host_update_validation():
    n, m, k = 4, 6, 2
    buf = (ctypes.c_float * (64 * 64))()
    base = ctypes.addressof(buf)
    acc, P, W = base, base + 4 * 256, base + 4 * 3000
    good = (ctypes.c_int32 * 4)(0, 2, 3, 5)
    EINVAL = 1
    assert _raw(acc, 4, ctypes.addressof(good), n, m, k, 0, P, 6, W, 4) == 0
    unsorted = (ctypes.c_int32 * 4)(0, 3, 2, 5)
    dup = (ctypes.c_int32 * 4)(0, 2, 2, 5)
    out_of_range = (ctypes.c_int32 * 4)(0, 2, 3, 6)
    for bad in (unsorted, dup, out_of_range):
        assert _raw(acc, 4, ctypes.addressof(bad), n, m, k, 0, P, 6, W, 4) == EINVAL
    assert _raw(acc, 3, ctypes.addressof(good), n, m, k, 0, P, 6, W, 4) == EINVAL  # ld < width
    assert _raw(acc, 4, ctypes.addressof(good), n, m, k, 0, P, 6, W, 4, step=0) == EINVAL
    assert _raw(acc, 4, ctypes.addressof(good), n, m, k, 0, P, 6, W, 4,
                scale=float("inf")) == EINVAL
    assert _raw(acc, 4, ctypes.addressof(good), n, m, k, 2, P, 6, W, 4) == EINVAL  # layout
    assert _raw(acc, 4, ctypes.addressof(good), n, m, k, 0, acc, 6, W, 4) == EINVAL  # overlap
    assert _raw(acc, 4, None, n, m, k, 0, P, 6, W, 4) == EINVAL
    assert _raw(None, 4, None, 0, m, k, 0, None, 6, None, 4) == 0  # n = 0: nothing to do
