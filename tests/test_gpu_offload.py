"""Parity of the offloaded optimizer's GPU parts and of the whole offloaded
step with the oracle, through the C ABI:

* zf_scatter_weights: W's unselected columns = the host-produced bf16
  columns, selected columns untouched, bit for bit; both layouts, the 16-byte
  and element paths, the source in device memory and in pinned host memory.
* swap against a full-state store inside the update pass (zf_adam_selected,
  zf_update_fused with store_* set): compact states of entering columns
  from the store, leaving columns' states written back to it, equal bit for
  bit to the oracle's swap_states followed by adam_selected (and
  pack_accumulate); the store in device memory and in pinned host memory.
* the runner's offload mode (deferred host update, synchronous and
  overlapped with the next interval) against OffloadOracle over several
  refreshes: selections, compact states, the whole store, the weights.
"""
import sys

import numpy as np
import pytest
import torch

import oracle as O
from tests._gpu import bf16_dev, bits_np, f32_dev, f32_np, same_bits
from workloads import derive_seed, gradient

pytestmark = pytest.mark.gpu

zf = pytest.importorskip("paper_2505_12242_amd")
HP = zf.AdamHparams(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.0)
LAYOUTS = [pytest.param(zf.ROW_MAJOR, id="rm"), pytest.param(zf.CHANNEL_MAJOR, id="cm")]


def T(a, layout):
    return a if layout == zf.ROW_MAJOR else np.ascontiguousarray(np.asarray(a).T)


def logical(a, layout):
    return a if layout == zf.ROW_MAJOR else np.ascontiguousarray(np.asarray(a).T)


def grad_bits(n, m, seed, sigma=1.5):
    g = torch.Generator().manual_seed(seed)
    s = torch.exp(sigma * torch.randn(m, generator=g, dtype=torch.float64))
    return bits_np(gradient(n, m, s, seed=seed))


def sel_dev(s: O.Selection):
    out = zf.Selection(s.m, s.k)
    out.sel_idx.copy_(torch.from_numpy(s.sel.astype(np.int32)))
    out.unsel_idx.copy_(torch.from_numpy(s.unsel.astype(np.int32)))
    out.mask.copy_(torch.from_numpy(s.mask.view(np.int64)))
    out.prefix.copy_(torch.from_numpy(s.prefix.astype(np.int32)))
    return out


def consts(t):
    return O.AdamConsts.at_step(HP.lr, HP.beta1, HP.beta2, HP.eps, HP.weight_decay, t)


def place(a, where):
    """fp32 / bf16-bits host array -> device tensor or pinned host tensor."""
    if a.dtype == np.uint16:
        t = torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16)
    else:
        t = torch.from_numpy(np.ascontiguousarray(a))
    if where == "device":
        return t.cuda()
    p = torch.empty(t.shape, dtype=t.dtype, pin_memory=True)
    p.copy_(t)
    return p


def host_np(t):
    if t.dtype == torch.bfloat16:
        return bits_np(t)
    return f32_np(t)


# ---------------------------------------------------------------- scatter

@pytest.mark.parametrize("n,m,ratio", [(1, 1, 0.0), (3, 7, 0.3), (64, 130, 0.1),
                                       (43, 77, 0.1), (4104, 40, 0.1), (16, 9, 1.0)])
@pytest.mark.parametrize("where", ["device", "pinned"])
@pytest.mark.parametrize("layout", LAYOUTS)
def test_scatter_weights(n, m, ratio, where, layout):
    rng = np.random.default_rng(n * 100 + m)
    sel = O.select_topk(rng.random(m).astype(np.float32), O.k_from_ratio(ratio, m))
    W = O.bf16_round((rng.standard_normal((n, m)) * 0.02).astype(np.float32))
    cols = O.bf16_round(rng.standard_normal((n, m - sel.k)).astype(np.float32))
    Wd = bf16_dev(T(W, layout))
    zf.scatter_weights(place(T(cols, layout), where), sel_dev(sel), Wd, layout=layout)
    torch.cuda.synchronize()
    want = W.copy()
    want[:, sel.unsel.astype(np.int64)] = cols
    assert np.array_equal(logical(bits_np(Wd), layout), want)


# ---------------------------------------------------------------- swap

def _store_arrays(rng, n, m):
    return ((rng.standard_normal((n, m)) * 0.02).astype(np.float32),
            (rng.standard_normal((n, m)) * 1e-3).astype(np.float32),
            (rng.random((n, m)) * 1e-5).astype(np.float32))


@pytest.mark.parametrize("n,m", [(33, 300), (8, 64), (4104, 70), (5, 9)])
@pytest.mark.parametrize("fused", [False, True])
@pytest.mark.parametrize("where", ["device", "pinned"])
@pytest.mark.parametrize("layout", LAYOUTS)
def test_swap_against_store(n, m, fused, where, layout):
    rng = np.random.default_rng(n + m)
    bits = grad_bits(n, m, derive_seed("swap", n, m))
    W = O.bf16_round((rng.standard_normal((n, m)) * 0.02).astype(np.float32))
    k_old, k_new = O.k_from_ratio(0.15, m), O.k_from_ratio(0.2, m)
    old = O.select_topk(rng.random(m).astype(np.float32), k_old)
    new = O.select_topk(rng.random(m).astype(np.float32), k_new)
    P, M, V = ((rng.standard_normal((n, k_old)) * s).astype(np.float32)
               for s in (0.02, 1e-3, 1e-5))
    V = np.abs(V)
    store = _store_arrays(rng, n, m)
    sd = [place(T(x, layout), where) for x in store]
    shape = (n, k_new) if layout == zf.ROW_MAJOR else (k_new, n)
    Pn = torch.full(shape, np.nan, device="cuda")
    Mn, Vn = torch.full_like(Pn, np.nan), torch.full_like(Pn, np.nan)
    Wd = bf16_dev(T(W, layout))
    src = zf.StateSource(prev=sel_dev(old), prev_master=f32_dev(T(P, layout)),
                         prev_exp_avg=f32_dev(T(M, layout)), prev_exp_avg_sq=f32_dev(T(V, layout)),
                         store_master=sd[0], store_exp_avg=sd[1], store_exp_avg_sq=sd[2])
    G = bf16_dev(T(bits, layout))
    if fused:
        ashape = (n, m - k_new) if layout == zf.ROW_MAJOR else (m - k_new, n)
        A = torch.full(ashape, np.nan, device="cuda")
        zf.update_fused(G, sel_dev(new), Pn, Mn, Vn, Wd, HP, 5, A, 1, 4, mode=zf.STATES_REMAP,
                        src=src, layout=layout)
    else:
        zf.adam_selected(G, sel_dev(new), Pn, Mn, Vn, Wd, HP, 5, mode=zf.STATES_REMAP, src=src,
                         layout=layout)
    torch.cuda.synchronize()
    P2, M2, V2, store2 = O.swap_states(old, new, P, M, V, store)
    Pw, Mw, Vw, wsel = O.adam_selected(bits, new.sel, P2, M2, V2, consts(5))
    for got, want in ((Pn, Pw), (Mn, Mw), (Vn, Vw)):
        assert same_bits(logical(f32_np(got), layout), want)
    for got, want in zip(sd, store2):
        assert same_bits(logical(host_np(got), layout), want)
    assert np.array_equal(logical(bits_np(Wd), layout)[:, new.sel.astype(np.int64)], wsel)
    if fused:
        assert same_bits(logical(f32_np(A), layout), O.pack_accumulate(bits, new.unsel, None, 1))
    # INIT from the store: every selected column swapped in, nothing written back
    Pi = torch.zeros(shape, device="cuda")
    Mi, Vi = torch.zeros_like(Pi), torch.zeros_like(Pi)
    zf.adam_selected(G, sel_dev(new), Pi, Mi, Vi, bf16_dev(T(W, layout)), HP, 1,
                     mode=zf.STATES_INIT,
                     src=zf.StateSource(store_master=sd[0], store_exp_avg=sd[1],
                                        store_exp_avg_sq=sd[2]), layout=layout)
    torch.cuda.synchronize()
    P3, M3, V3, _ = O.swap_states(None, new, None, None, None, store2)
    Pw, Mw, Vw, _ = O.adam_selected(bits, new.sel, P3, M3, V3, consts(1))
    for got, want in ((Pi, Pw), (Mi, Mw), (Vi, Vw)):
        assert same_bits(logical(f32_np(got), layout), want)
    for got, want in zip(sd, store2):
        assert same_bits(logical(host_np(got), layout), want)


def test_store_overlapping_an_output_is_rejected():
    n, m = 8, 64
    new = O.select_topk(np.arange(m, dtype=np.float32), 8)
    buf = torch.zeros(3 * n * m + 64, device="cuda")
    P = buf[: n * 8].view(n, 8)
    src = zf.StateSource(store_master=buf[: n * m].view(n, m),  # overlaps P
                         store_exp_avg=buf[n * m: 2 * n * m].view(n, m),
                         store_exp_avg_sq=buf[2 * n * m: 3 * n * m].view(n, m))
    with pytest.raises(zf.ZfError, match="invalid argument"):
        zf.adam_selected(torch.zeros(n, m, dtype=torch.bfloat16, device="cuda"), sel_dev(new),
                         P, torch.zeros(n, 8, device="cuda"), torch.zeros(n, 8, device="cuda"),
                         torch.zeros(n, m, dtype=torch.bfloat16, device="cuda"), HP, 1,
                         mode=zf.STATES_INIT, src=src)


# ---------------------------------------------------------------- whole step

SET = [(264, 300), (4104, 70), (43, 77), (128, 1000), (16, 3)]


def _inputs(shapes, T_, seed, layout, dev):
    slots, host = [], []
    for t in range(1, T_ + 1):
        ds, hs = [], []
        for q, (n, m) in enumerate(shapes):
            g = torch.Generator().manual_seed(derive_seed(seed, q, "s") & 0x7fffffff)
            base = torch.exp(1.5 * torch.randn(m, generator=g, dtype=torch.float64))
            # a few channels swap places from step to step: selections change
            jit = torch.exp(0.3 * torch.randn(m, generator=torch.Generator().manual_seed(
                derive_seed(seed, q, "j", t) & 0x7fffffff), dtype=torch.float64))
            gr = gradient(n, m, base * jit, derive_seed(seed, q, "g", t), device=dev)
            hs.append(bits_np(gr))
            ds.append(gr if layout == zf.ROW_MAJOR else gr.t().contiguous())
        slots.append(ds)
        host.append(hs)
    weights, w0 = [], []
    for q, (n, m) in enumerate(shapes):
        g = torch.Generator().manual_seed(derive_seed(seed, q, "w") & 0x7fffffff)
        w = (0.02 * torch.randn(n, m, generator=g)).to(torch.bfloat16)
        w0.append(bits_np(w))
        weights.append((w if layout == zf.ROW_MAJOR else w.t().contiguous()).to(dev))
    return slots, host, weights, w0


@pytest.mark.timeout(600)
@pytest.mark.parametrize("overlap", [False, True])
@pytest.mark.parametrize("R,S,W", [(2, 2, 0), (6, 2, 0), (6, 2, 3)])
@pytest.mark.parametrize("layout", LAYOUTS)
def test_offloaded_steps_match_oracle(layout, R, S, W, overlap):
    """W > 0: the first W steps are synchronous (one-step intervals, each
    deferred update landing before the next step)."""
    T_ = 8
    dev = torch.device("cuda")
    slots, host, weights, w0 = _inputs(SET, T_, 21, layout, dev)
    runner = zf.SelectiveUpdateRunner(SET, 0.1, HP, R, S, slots, weights, device=dev,
                                      layout=layout, offload=True, overlap=overlap,
                                      host_threads=4, warmup=W)
    orcs = [O.OffloadOracle(O.widen(w0[q]), w0[q], 0.1, HP.lr, HP.beta1, HP.beta2, HP.eps,
                            HP.weight_decay, R, S, warmup=W) for q in range(len(SET))]
    changed = 0
    for t in range(1, T_ + 1):
        print(f"# offload layout={layout} R={R} S={S} W={W} overlap={overlap} step {t}",
              file=sys.stderr, flush=True)
        prev = [s.sel_idx.cpu().numpy().copy() for s in runner.selection] if t > 1 else None
        kind = runner.step()
        outs = [o.step(host[t - 1][q]) for q, o in enumerate(orcs)]
        ok = outs[0]["kind"]
        assert (kind.refresh, kind.step_in_interval, kind.interval_end) == \
            (ok.refresh, ok.step_in_interval, ok.interval_end)
        if t % 2 == 0 or t == T_:  # compare at a few synchronised points
            runner.sync()
            for q, o in enumerate(orcs):
                assert np.array_equal(runner.selection[q].sel_idx.cpu().numpy(), o.sel.sel)
                for got, want in zip(runner.state[q], (o.P, o.M, o.V)):
                    assert same_bits(logical(f32_np(got), layout), want), (q, t)
                for got, want in zip(runner.store[q], o.store):
                    assert same_bits(logical(got.numpy(), layout), want), (q, t)
                assert np.array_equal(logical(bits_np(runner.weights[q]), layout), o.W), (q, t)
        if kind.refresh and prev is not None:
            changed += sum(int(np.setdiff1d(s.sel_idx.cpu().numpy(), p0).size)
                           for s, p0 in zip(runner.selection, prev))
    assert runner.th == orcs[0].th
    assert changed > 0  # selections really changed: swaps were exercised
    runner.close()


@pytest.mark.timeout(600)
@pytest.mark.parametrize("overlap", [False, True])
def test_zen_auto_triggers_the_deferred_update(overlap):
    """Zen-auto with the offloaded optimizer (channel-major): the trigger
    ends the interval and starts the deferred host update.  Against
    ZenAutoOracle over OffloadOracles: interval ends, totals, and at
    synchronised points the compact states, the whole store and W, bit for
    bit; tau sits between the ratios observed after one and after several
    accumulated steps, so intervals end early."""
    import math
    layout, R, S_max, T_ = zf.CHANNEL_MAJOR, 16, 6, 10
    dev = torch.device("cuda")
    slots, host, weights, w0 = _inputs(SET, T_, 23, layout, dev)

    def oracles(tau):
        return O.ZenAutoOracle([O.OffloadOracle(O.widen(w0[q]), w0[q], 0.1, HP.lr, HP.beta1,
                                                HP.beta2, HP.eps, HP.weight_decay, R, S_max)
                                for q in range(len(SET))], R, S_max, tau)

    probe = oracles(math.inf)
    ratios = []
    for t in range(T_):
        tot = probe.step(host[t])["totals"]
        ratios.append((tot.sum_acc / tot.u) / (tot.sum_sel / tot.k))
    tau = math.sqrt(min(ratios[:2]) * max(ratios[2:S_max]))
    za = oracles(tau)
    runner = zf.SelectiveUpdateRunner(SET, 0.1, HP, R, S_max, slots, weights, device=dev,
                                      layout=layout, zen_tau=tau, offload=True, overlap=overlap,
                                      host_threads=4)
    ends = []
    for t in range(1, T_ + 1):
        print(f"# zen+offload overlap={overlap} step {t}", file=sys.stderr, flush=True)
        kind = runner.step()
        ref = za.step(host[t - 1])
        assert (kind.refresh, kind.step_in_interval, kind.interval_end) == \
            (ref["refresh"], ref["step_in_interval"], ref["interval_end"]), t
        got, want = runner.last_totals, ref["totals"]
        assert abs(got.sum_acc - want.sum_acc) <= 1e-9 * want.sum_acc
        assert got.trigger == want.trigger
        ends.append(kind.interval_end)
        if t % 3 == 0 or t == T_:
            runner.sync()
            for q, o in enumerate(za.orcs):
                for g_, w_ in zip(runner.state[q], (o.P, o.M, o.V)):
                    assert same_bits(logical(f32_np(g_), layout), w_), (q, t)
                for g_, w_ in zip(runner.store[q], o.store):
                    assert same_bits(logical(g_.numpy(), layout), w_), (q, t)
                assert np.array_equal(logical(bits_np(runner.weights[q]), layout), o.W), (q, t)
    assert any(ends) and not all(ends)
    assert runner.th == za.orcs[0].th == sum(ends)
    runner.close()


@pytest.mark.parametrize("layout", LAYOUTS)
def test_remap_with_store_requires_previous_states(layout):
    """With a store, a remap reads the previous compact states for the
    columns that leave the selection even when no column is selected now
    (k = 0): they are required, and a k = 0 remap swaps every previously
    selected column out."""
    n, m = 16, 40
    rng = np.random.default_rng(7)
    old = O.select_topk(rng.random(m).astype(np.float32), 6)
    new = O.select_topk(rng.random(m).astype(np.float32), 0)
    store = _store_arrays(rng, n, m)
    sd = [place(T(x, layout), "device") for x in store]
    P, M, V = ((rng.standard_normal((n, 6)) * s).astype(np.float32) for s in (0.02, 1e-3, 1e-5))
    V = np.abs(V)
    shape = (n, 0) if layout == zf.ROW_MAJOR else (0, n)
    empty = [torch.empty(shape, device="cuda") for _ in range(3)]
    Wd = bf16_dev(T(O.bf16_round(rng.standard_normal((n, m)).astype(np.float32)), layout))
    G = bf16_dev(T(grad_bits(n, m, 3), layout))
    no_prev = zf.StateSource(prev=sel_dev(old), store_master=sd[0], store_exp_avg=sd[1],
                             store_exp_avg_sq=sd[2])
    with pytest.raises(zf.ZfError):
        zf.adam_selected(G, sel_dev(new), *empty, Wd, HP, 2, mode=zf.STATES_REMAP, src=no_prev,
                         layout=layout)
    src = zf.StateSource(prev=sel_dev(old), prev_master=f32_dev(T(P, layout)),
                         prev_exp_avg=f32_dev(T(M, layout)), prev_exp_avg_sq=f32_dev(T(V, layout)),
                         store_master=sd[0], store_exp_avg=sd[1], store_exp_avg_sq=sd[2])
    zf.adam_selected(G, sel_dev(new), *empty, Wd, HP, 2, mode=zf.STATES_REMAP, src=src,
                     layout=layout)
    torch.cuda.synchronize()
    _, _, _, store2 = O.swap_states(old, new, P, M, V, store)
    for got, want in zip(sd, store2):
        assert same_bits(T(f32_np(got), layout), want)
