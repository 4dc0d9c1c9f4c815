"""The refresh that does not wait for the host (offloaded optimizer), through
the C ABI:

* zf_plan_update_pending: a remap + fused update against the full-state
  store in which each column entering the selection first takes the
  deferred step its store column still owes (from the previous interval's
  packed sums) equals, bit for bit, the oracle's order -- deferred_adam
  landing in the store, then swap_states and adam_selected -- and leaves
  the entering columns' store columns as they were (only read), so that the
  host update applied afterwards gives the synchronous order's store;
* zf_plan_scatter_weights_skip_prev: the write-back under the previous
  selection leaves the refreshed selection's columns alone;
* the runner with refresh_pending on and off against OffloadOracle over
  several refreshes, compared only after refresh steps and at the end, so
  that the held-back host updates, the staged write-backs and the skipping
  write-back all run inside the pipeline.
"""
import sys

import numpy as np
import pytest
import torch

import oracle as O
from tests._gpu import bf16_dev, bits_np, f32_dev, f32_np, same_bits
from tests.test_gpu_offload import (HP, LAYOUTS, SET, T, _inputs, _store_arrays, consts,
                                    grad_bits, host_np, logical, place, sel_dev)
from workloads import derive_seed, gradient

pytestmark = pytest.mark.gpu

zf = pytest.importorskip("paper_2505_12242_amd")


def _nan(shape):
    return torch.full(shape, np.nan, device="cuda")


@pytest.mark.parametrize("n,m", [(33, 300), (8, 64), (4104, 70), (5, 9), (256, 1001)])
@pytest.mark.parametrize("where", ["device", "pinned"])
@pytest.mark.parametrize("layout", LAYOUTS)
def test_update_pending_equals_host_update_then_refresh(n, m, where, layout):
    print(f"# pending n={n} m={m} where={where} layout={layout}", file=sys.stderr, flush=True)
    rng = np.random.default_rng(derive_seed("pend", n, m))
    k = O.k_from_ratio(0.25, m)
    old = O.select_topk(rng.random(m).astype(np.float32), k)
    new = O.select_topk(rng.random(m).astype(np.float32), k)
    assert np.setdiff1d(new.sel, old.sel).size > 0  # some columns enter
    bits = grad_bits(n, m, derive_seed("pend-g", n, m))
    W = O.bf16_round((rng.standard_normal((n, m)) * 0.02).astype(np.float32))
    P, M, V = ((rng.standard_normal((n, k)) * s).astype(np.float32) for s in (0.02, 1e-3, 1e-5))
    V = np.abs(V)
    store = _store_arrays(rng, n, m)
    Apend = (rng.standard_normal((n, m - k)) * 0.05).astype(np.float32)
    pend_step, pend_scale, step = 3, float(np.float32(1.0 / 3.0)), 11

    rm = layout == zf.ROW_MAJOR
    sd = [place(T(x, layout), where) for x in store]
    Pn, Mn, Vn = (_nan((n, k) if rm else (k, n)) for _ in range(3))
    A = _nan((n, m - k) if rm else (m - k, n))
    Wd = bf16_dev(T(W, layout))
    src = zf.StateSource(prev=sel_dev(old), prev_master=f32_dev(T(P, layout)),
                         prev_exp_avg=f32_dev(T(M, layout)), prev_exp_avg_sq=f32_dev(T(V, layout)),
                         store_master=sd[0], store_exp_avg=sd[1], store_exp_avg_sq=sd[2],
                         pend_acc=f32_dev(T(Apend, layout)))
    plan = zf.Plan([zf.MatrixBuffers(grad=bf16_dev(T(bits, layout)), k=k, sel=sel_dev(new),
                                     weight=Wd, master=Pn, exp_avg=Mn, exp_avg_sq=Vn, acc=A,
                                     src=src, layout=layout)])
    plan.update_pending(HP, step, 4, pend_step, pend_scale)
    torch.cuda.synchronize()

    # the synchronous order: the host update lands in the store, then a plain refresh
    store1, _ = O.deferred_adam(Apend, old.unsel, pend_scale, store, consts(pend_step))
    P2, M2, V2, store2 = O.swap_states(old, new, P, M, V, store1)
    Pw, Mw, Vw, wsel = O.adam_selected(bits, new.sel, P2, M2, V2, consts(step))
    for got, want in ((Pn, Pw), (Mn, Mw), (Vn, Vw)):
        assert same_bits(logical(f32_np(got), layout), want)
    Wgot = logical(bits_np(Wd), layout)
    assert np.array_equal(Wgot[:, new.sel.astype(np.int64)], wsel)
    assert np.array_equal(Wgot[:, new.unsel.astype(np.int64)], W[:, new.unsel.astype(np.int64)])
    assert same_bits(logical(f32_np(A), layout), O.pack_accumulate(bits, new.unsel, None, 1))
    # the store: leaving columns written back, entering columns only read ...
    got = [logical(host_np(x), layout) for x in sd]
    _, _, _, swapped = O.swap_states(old, new, P, M, V, store)
    for g, want in zip(got, swapped):
        assert same_bits(g, want)
    # ... so the host update applied afterwards reaches the synchronous store
    after, _ = O.deferred_adam(Apend, old.unsel, pend_scale, got, consts(pend_step))
    for g, want in zip(after, store2):
        assert same_bits(g, want)
    plan.close()


def test_update_pending_needs_the_store_and_the_sums():
    n, m, k = 8, 64, 16
    rng = np.random.default_rng(5)
    old = O.select_topk(rng.random(m).astype(np.float32), k)
    new = O.select_topk(rng.random(m).astype(np.float32), k)
    P = f32_dev(np.zeros((n, k), np.float32))
    base = dict(grad=bf16_dev(np.zeros((n, m), np.uint16)), k=k, sel=sel_dev(new),
                weight=bf16_dev(np.zeros((n, m), np.uint16)), master=_nan((n, k)),
                exp_avg=_nan((n, k)), exp_avg_sq=_nan((n, k)), acc=_nan((n, m - k)))
    store = [torch.zeros(n, m, device="cuda") for _ in range(3)]
    no_sums = zf.StateSource(prev=sel_dev(old), prev_master=P, prev_exp_avg=P.clone(),
                             prev_exp_avg_sq=P.clone(), store_master=store[0],
                             store_exp_avg=store[1], store_exp_avg_sq=store[2])
    plan = zf.Plan([zf.MatrixBuffers(src=no_sums, **base)])
    with pytest.raises(RuntimeError):
        plan.update_pending(HP, 2, 4, 1, 1.0)
    plan.close()
    no_store = zf.StateSource(prev=sel_dev(old), prev_master=P, prev_exp_avg=P.clone(),
                              prev_exp_avg_sq=P.clone(), pend_acc=_nan((n, m - k)))
    plan = zf.Plan([zf.MatrixBuffers(src=no_store, **base)])
    with pytest.raises(RuntimeError):
        plan.update_pending(HP, 2, 4, 1, 1.0)
    plan.close()
    # the sums overlapping a buffer the call writes
    acc = base["acc"]
    ok_src = zf.StateSource(prev=sel_dev(old), prev_master=P, prev_exp_avg=P.clone(),
                            prev_exp_avg_sq=P.clone(), store_master=store[0],
                            store_exp_avg=store[1], store_exp_avg_sq=store[2], pend_acc=acc)
    plan = zf.Plan([zf.MatrixBuffers(src=ok_src, **base)])
    with pytest.raises(RuntimeError):
        plan.update_pending(HP, 2, 4, 1, 1.0)
    plan.close()


@pytest.mark.parametrize("n,m", [(43, 77), (4104, 40), (8, 1000), (3, 7)])
@pytest.mark.parametrize("layout", LAYOUTS)
def test_scatter_weights_skip_prev(n, m, layout):
    rng = np.random.default_rng(derive_seed("skip", n, m))
    k = O.k_from_ratio(0.3, m)
    old = O.select_topk(rng.random(m).astype(np.float32), k)
    new = O.select_topk(rng.random(m).astype(np.float32), k)
    W = O.bf16_round((rng.standard_normal((n, m)) * 0.02).astype(np.float32))
    cols = O.bf16_round(rng.standard_normal((n, m - k)).astype(np.float32))
    Wd = bf16_dev(T(W, layout))
    plan = zf.Plan([zf.MatrixBuffers(grad=bf16_dev(T(np.zeros((n, m), np.uint16), layout)), k=k,
                                     sel=sel_dev(old), weight=Wd,
                                     src=zf.StateSource(prev=sel_dev(new)), layout=layout,
                                     weight_cols=place(T(cols, layout), "device"))])
    plan.scatter_weights_skip_prev()
    torch.cuda.synchronize()
    want = W.copy()
    for u, j in enumerate(old.unsel.tolist()):
        if not new.mask[j >> 6] >> np.uint64(j & 63) & np.uint64(1):
            want[:, j] = cols[:, u]
    assert np.array_equal(logical(bits_np(Wd), layout), want)
    plan.close()


@pytest.mark.timeout(600)
@pytest.mark.parametrize("pending", [True, False])
@pytest.mark.parametrize("R,S,W", [(2, 2, 0), (4, 2, 0), (1, 1, 0), (4, 4, 0), (4, 2, 3)])
@pytest.mark.parametrize("layout", LAYOUTS)
def test_pipelined_refreshes_match_oracle(layout, R, S, W, pending):
    """W > 0: the first W steps are synchronous (their refreshes wait)."""
    T_ = 13
    dev = torch.device("cuda")
    slots, host, weights, w0 = _inputs(SET, T_, 23, layout, dev)
    runner = zf.SelectiveUpdateRunner(SET, 0.1, HP, R, S, slots, weights, device=dev,
                                      layout=layout, offload=True, overlap=True,
                                      host_threads=4, refresh_pending=pending, warmup=W)
    orcs = [O.OffloadOracle(O.widen(w0[q]), w0[q], 0.1, HP.lr, HP.beta1, HP.beta2, HP.eps,
                            HP.weight_decay, R, S, warmup=W) for q in range(len(SET))]
    for t in range(1, T_ + 1):
        print(f"# pipelined layout={layout} R={R} S={S} W={W} pending={pending} step {t}",
              file=sys.stderr, flush=True)
        runner.step()
        for q, o in enumerate(orcs):
            o.step(host[t - 1][q])
        if t in (7, T_):
            runner.sync()
            for q, o in enumerate(orcs):
                assert np.array_equal(runner.selection[q].sel_idx.cpu().numpy(), o.sel.sel)
                for got, want in zip(runner.state[q], (o.P, o.M, o.V)):
                    assert same_bits(logical(f32_np(got), layout), want), (q, t)
                for got, want in zip(runner.store[q], o.store):
                    assert same_bits(logical(got.numpy(), layout), want), (q, t)
                assert np.array_equal(logical(bits_np(runner.weights[q]), layout), o.W), (q, t)
    assert runner.th == orcs[0].th
    assert (runner.pending_refreshes > 0) == pending
    runner.close()


@pytest.mark.parametrize("n,m", [(33, 300), (4104, 70)])
@pytest.mark.parametrize("layout", LAYOUTS)
def test_update_zen_pending_equals_zen_refresh_on_the_updated_store(n, m, layout):
    """zf_plan_update_zen_pending against zf_plan_update_zen (remap) on a
    store that already holds the deferred update (the oracle's): compact
    states, W, packed buffer, store, both statistics vectors and the totals
    bit for bit."""
    print(f"# zen pending n={n} m={m} layout={layout}", file=sys.stderr, flush=True)
    rng = np.random.default_rng(derive_seed("zen-pend", n, m))
    k = O.k_from_ratio(0.25, m)
    old = O.select_topk(rng.random(m).astype(np.float32), k)
    new = O.select_topk(rng.random(m).astype(np.float32), k)
    bits = grad_bits(n, m, derive_seed("zen-pend-g", n, m))
    W = O.bf16_round((rng.standard_normal((n, m)) * 0.02).astype(np.float32))
    P, M, V = ((rng.standard_normal((n, k)) * s).astype(np.float32) for s in (0.02, 1e-3, 1e-5))
    V = np.abs(V)
    store = _store_arrays(rng, n, m)
    Apend = (rng.standard_normal((n, m - k)) * 0.05).astype(np.float32)
    pend_step, pend_scale, step, tau = 2, float(np.float32(0.5)), 7, 1.0
    store1, _ = O.deferred_adam(Apend, old.unsel, pend_scale, store, consts(pend_step))
    rm = layout == zf.ROW_MAJOR

    def run(pending):
        sd = [place(T(x, layout), "pinned") for x in (store if pending else store1)]
        bufs = dict(master=_nan((n, k) if rm else (k, n)), exp_avg=_nan((n, k) if rm else (k, n)),
                    exp_avg_sq=_nan((n, k) if rm else (k, n)),
                    acc=_nan((n, m - k) if rm else (m - k, n)),
                    sel_sq=torch.full((k,), np.nan, device="cuda"),
                    acc_sq=torch.full((m - k,), np.nan, device="cuda"))
        Wd = bf16_dev(T(W, layout))
        src = zf.StateSource(prev=sel_dev(old), prev_master=f32_dev(T(P, layout)),
                             prev_exp_avg=f32_dev(T(M, layout)),
                             prev_exp_avg_sq=f32_dev(T(V, layout)),
                             store_master=sd[0], store_exp_avg=sd[1], store_exp_avg_sq=sd[2],
                             pend_acc=f32_dev(T(Apend, layout)) if pending else None)
        plan = zf.Plan([zf.MatrixBuffers(grad=bf16_dev(T(bits, layout)), k=k, sel=sel_dev(new),
                                         weight=Wd, src=src, layout=layout, **bufs)])
        totals = torch.zeros(zf.ZEN_TOTALS_BYTES // 8, dtype=torch.int64, device="cuda")
        if pending:
            plan.update_zen_pending(HP, step, 4, pend_step, pend_scale, tau, totals)
        else:
            plan.update_zen(HP, step, zf.STATES_REMAP, 1, 4, tau, totals)
        torch.cuda.synchronize()
        out = [bufs[x].cpu().numpy() for x in ("master", "exp_avg", "exp_avg_sq", "acc",
                                                "sel_sq", "acc_sq")]
        out.append(bits_np(Wd))
        out.append(totals.cpu().numpy())
        plan.close()
        return out, [host_np(x) for x in sd]

    got, got_store = run(True)
    want, want_store = run(False)
    for g, w in zip(got, want):
        assert g.tobytes() == w.tobytes()
    # the pending run left the entering columns' store columns as they were;
    # the host update applied afterwards reaches the other run's store
    after, _ = O.deferred_adam(Apend, old.unsel, pend_scale,
                               [logical(x, layout) for x in got_store], consts(pend_step))
    for g, w in zip(after, want_store):
        assert same_bits(g, logical(w, layout))


@pytest.mark.timeout(600)
@pytest.mark.parametrize("layout", LAYOUTS)
def test_zen_auto_pipelined_refreshes_match_oracle(layout):
    """Zen-auto with the offloaded optimizer, refreshes every 4 steps: the
    forced interval end before each refresh is taken over by the refresh
    (zf_plan_update_zen_pending); interval ends, totals, and after refresh
    steps and at the end the compact states, the whole store and W against
    ZenAutoOracle over OffloadOracles, bit for bit."""
    import math
    R, S_max, T_ = 4, 4, 13
    dev = torch.device("cuda")
    slots, host, weights, w0 = _inputs(SET, T_, 29, layout, dev)

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
                                      layout=layout, zen_tau=tau, offload=True, overlap=True,
                                      host_threads=4)
    for t in range(1, T_ + 1):
        print(f"# zen pipelined layout={layout} step {t}", file=sys.stderr, flush=True)
        kind = runner.step()
        ref = za.step(host[t - 1])
        assert (kind.refresh, kind.step_in_interval, kind.interval_end) == \
            (ref["refresh"], ref["step_in_interval"], ref["interval_end"]), t
        assert runner.last_totals.trigger == ref["totals"].trigger
        if t in (7, T_):
            runner.sync()
            for q, o in enumerate(za.orcs):
                for g_, w_ in zip(runner.state[q], (o.P, o.M, o.V)):
                    assert same_bits(logical(f32_np(g_), layout), w_), (q, t)
                for g_, w_ in zip(runner.store[q], o.store):
                    assert same_bits(logical(g_.numpy(), layout), w_), (q, t)
                assert np.array_equal(logical(bits_np(runner.weights[q]), layout), o.W), (q, t)
    assert runner.pending_refreshes > 0
    assert runner.th == za.orcs[0].th
    runner.close()


def _layer_inputs(T_, layout, dev):
    """One Llama-2-7B decoder layer's gradients for T_ steps (device) and its
    bf16 weights, in `layout`."""
    from workloads.configs import get_workload, shapes as wl_shapes
    shp = wl_shapes(get_workload("llama2-7b-layer").matrices)
    slots = []
    for t in range(1, T_ + 1):
        row = []
        for q, (n, m) in enumerate(shp):
            s = torch.exp(1.5 * torch.randn(m, generator=torch.Generator().manual_seed(
                derive_seed("layer-s", q) & 0x7fffffff), dtype=torch.float64))
            jit = torch.exp(0.3 * torch.randn(m, generator=torch.Generator().manual_seed(
                derive_seed("layer-j", q, t) & 0x7fffffff), dtype=torch.float64))
            g = gradient(n, m, s * jit, derive_seed("layer-g", q, t), device=dev)
            row.append(g if layout == zf.ROW_MAJOR else g.t().contiguous())
        slots.append(row)
    w = []
    for q, (n, m) in enumerate(shp):
        x = (0.02 * torch.randn(n, m, generator=torch.Generator().manual_seed(q))).to(torch.bfloat16)
        w.append((x if layout == zf.ROW_MAJOR else x.t().contiguous()).to(dev))
    return shp, slots, w


@pytest.mark.timeout(900)
@pytest.mark.parametrize("busy", [False, True])
@pytest.mark.parametrize("layout", LAYOUTS)
def test_layer_size_pipeline_equals_synchronous(layout, busy):
    """A whole 7B decoder layer (202 M parameters): the overlapped runner with
    pipelined refreshes against the synchronous runner over the same 10
    steps (R = 4, S = 2: refreshes at steps 1, 5 and 9, the last two taking
    over the interval that ends right before them), every buffer compared
    bit for bit at the end.  At this size the host update
    (~30 ms) outlasts several device steps: with busy=False the hand-overs
    wait for it; with busy=True a stand-in compute of ~8 ms per step on the
    same stream lets it finish between steps, so the staged write-backs land
    at later boundaries."""
    T_, R, S = 10, 4, 2
    dev = torch.device("cuda")
    shp, slots, w = _layer_inputs(T_, layout, dev)
    a = torch.randn(4096, 4096, device=dev, dtype=torch.bfloat16)
    b = torch.randn(4096, 4096, device=dev, dtype=torch.bfloat16)
    c = torch.empty_like(a)
    runs = []
    for overlap in (True, False):
        weights = [x.clone() for x in w]
        runner = zf.SelectiveUpdateRunner(shp, 0.1, HP, R, S, slots, weights, device=dev,
                                          layout=layout, offload=True, overlap=overlap,
                                          host_threads=8)
        for t in range(1, T_ + 1):
            print(f"# layer pipeline layout={layout} busy={busy} overlap={overlap} step {t}",
                  file=sys.stderr, flush=True)
            if busy and overlap:
                for _ in range(60):
                    torch.mm(a, b, out=c)
            runner.step()
        runner.sync()
        if overlap:
            assert runner.pending_refreshes == 2  # steps 5 and 9
        out = []
        for q in range(len(shp)):
            out.append(runner.selection[q].sel_idx.cpu().numpy())
            out.extend(x.cpu().numpy() for x in runner.state[q])
            out.extend(x.numpy().copy() for x in runner.store[q])
            out.append(bits_np(runner.weights[q]))
        runs.append(out)
        runner.close()
        del runner, weights
        torch.cuda.synchronize()
    assert len(runs[0]) == len(runs[1])
    for i, (g, want) in enumerate(zip(*runs)):
        assert g.shape == want.shape and g.dtype == want.dtype, i
        assert np.array_equal(np.ascontiguousarray(g).view(np.uint8),
                              np.ascontiguousarray(want).view(np.uint8)), i
