"""Adam at its numerical edges on the host side (no GPU).

* The edge inputs shared with the device test (tests/test_gpu_adam_edges.py)
  do reach every regime that test is about: zero, eps-sized, subnormal-square
  and overflowing-square gradients, subnormal and zero moments, NaN results
  when moments are infinite.
* The deferred host update (zf_host_adam_unselected, the offloaded
  optimizer's step of the unselected columns: Asynchronous Offloading
  Workflow; Implementation, "Concurrent CPU-side Optimizer") equals the
  oracle's deferred_adam bit for bit on packed sums and store states drawn
  over the same classes (NaN matches NaN), both layouts, 1 and several
  threads, with and without decay, at steps 1 and 1000.
"""
import numpy as np
import pytest
import torch

import oracle as O
from tests._edges import bf16_as_f32, first_mismatch, inputs, same_nan_aware
from workloads import derive_seed, edge_f32, sprinkle_nonfinite

zf = pytest.importorskip("paper_2505_12242_amd")


def test_edge_inputs_reach_every_class():
    n, m, ratio = 72, 300, 0.3
    G, sel, P, Mo, V, W, A, master = inputs(n, m, ratio, 1, False)
    g = np.abs(bf16_as_f32(G))
    assert (g == 0).sum() > 100
    assert ((g > 1e-9) & (g < 1.2e-7)).sum() > 100
    assert ((g > 0) & (g < 2.0 ** -64)).sum() > 100
    assert ((g > 0) & (g < np.finfo(np.float32).tiny)).sum() > 100  # bf16 subnormals
    assert (g >= 2.0 ** 64).sum() > 100
    assert ((V > 0) & (V < np.finfo(np.float32).tiny)).sum() > 100
    assert (V == 0).sum() > 100 and (Mo == 0).sum() > 100 and np.signbit(V).sum() > 0
    c = O.AdamConsts.at_step(1e-3, 0.9, 0.999, 1e-8, 0.0, 1)
    with np.errstate(all="ignore"):
        Pw, Mw, Vw, _ = O.adam_selected(G, sel.sel, P, Mo, V, c)
        gs = bf16_as_f32(G[:, sel.sel.astype(np.int64)])
        assert np.isinf(gs * gs).sum() > 100  # g * g overflows
        sq = c.C2 * (gs * gs)
        assert ((sq > 0) & (sq < np.finfo(np.float32).tiny)).sum() > 10  # subnormal C2 * g^2
        assert ((gs != 0) & (sq == 0)).sum() > 10  # C2 * g^2 underflows to zero
    assert np.isinf(Vw).sum() > 0
    G2, sel2, P2, M2, V2, *_ = inputs(n, m, ratio, 1, True)
    with np.errstate(all="ignore"):
        Pn, *_ = O.adam_selected(G2, sel2.sel, P2, M2, V2, c)
    assert np.isnan(Pn).sum() > 0


def _host(x, layout, pad, dtype=torch.float32):
    x = x if layout == zf.ROW_MAJOR else np.ascontiguousarray(np.asarray(x).T)
    r, c = x.shape
    buf = torch.zeros(r, c + pad, dtype=dtype)
    if dtype == torch.float32:
        buf[:, :c] = torch.from_numpy(np.ascontiguousarray(x, np.float32))
    return buf[:, :c]


def _logical(t, layout):
    a = t.numpy() if t.dtype != torch.bfloat16 else t.view(torch.int16).numpy().view(np.uint16)
    return a if layout == zf.ROW_MAJOR else np.ascontiguousarray(a.T)


@pytest.mark.parametrize("nonfinite", [False, True], ids=["finite", "inf-moments"])
@pytest.mark.parametrize("step", [1, 1000])
@pytest.mark.parametrize("wd", [0.0, 0.01])
@pytest.mark.parametrize("scale", [1.0, 0.25, 1.0 / 3.0])
@pytest.mark.parametrize("threads", [1, 4])
@pytest.mark.parametrize("layout", [zf.ROW_MAJOR, zf.CHANNEL_MAJOR], ids=["rm", "cm"])
def test_host_update_edges(layout, threads, scale, wd, step, nonfinite):
    n, m, ratio = 40, 260, 0.2
    seed = derive_seed("host-edges", step, int(nonfinite))
    rng = np.random.default_rng(seed)
    sel = O.select_topk(rng.random(m).astype(np.float32), O.k_from_ratio(ratio, m))
    u = m - sel.k
    A = edge_f32((n, u), derive_seed("a", seed), "sum")
    SP = edge_f32((n, m), derive_seed("p", seed), "master")
    SM = edge_f32((n, m), derive_seed("m", seed), "first")
    SV = edge_f32((n, m), derive_seed("v", seed), "second")
    if nonfinite:
        SM, SV = sprinkle_nonfinite(SM, SV, seed)
    scale = float(np.float32(scale))
    hp = zf.AdamHparams(lr=1e-3, weight_decay=wd)
    c = O.AdamConsts.at_step(hp.lr, hp.beta1, hp.beta2, hp.eps, hp.weight_decay, step)
    with np.errstate(all="ignore"):
        (WP, WM, WV), Ww = O.deferred_adam(A, sel.unsel, scale, (SP, SM, SV), c)
    acc = _host(A, layout, 3)
    P, Mt, V = (_host(x, layout, 5) for x in (SP, SM, SV))
    wcols = _host(np.zeros((n, u), np.float32), layout, 2, torch.bfloat16)
    zf.host_adam_unselected(acc, torch.from_numpy(sel.unsel.astype(np.int32)), n, m, sel.k,
                            scale, P, Mt, V, wcols, hp, step=step, layout=layout,
                            nthreads=threads)
    for name, got, want in (("P", P, WP), ("M", Mt, WM), ("V", V, WV)):
        g = _logical(got, layout)
        assert same_nan_aware(g, want), (name, first_mismatch(g, want))
    wg = bf16_as_f32(_logical(wcols, layout))
    assert same_nan_aware(wg, bf16_as_f32(Ww)), ("W", first_mismatch(wg, bf16_as_f32(Ww)))
