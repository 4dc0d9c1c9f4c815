"""Parity of Zen-auto (the adaptive accumulation interval, Zero-stall
Pipeline "Hyperparameter Auto-tuning") on the GPU with the oracle's
ZenAutoOracle, through zf_plan_update_zen, in both layouts (statistics fused
into the update in the channel-major layout, a separate pass in the
row-major layout):

* per channel: the selected channels' squared gradient norms and the
  accumulated channels' squared norms, within 1e-5 relative (both sides sum
  exact squares in fp64 and round once to fp32, in different orders);
* set-wide: the sums of channel norms within 1e-9 relative (fp64 sums of
  ~10^3 terms in different orders), k and u exactly, and the trigger equal
  wherever the oracle's comparison is not within 1e-9 of a tie;
* the schedule it drives (interval lengths, ends, hand-over scale) and every
  state, packed buffer, weight and hand-over bit for bit, as in the fixed
  schedule;
* channel-major with deferred packing (zf_plan_update_zen_deferred): the
  unselected channels' statistics from the interval's kept gradients summed
  again at every step; the same checks, nothing packed.

Shapes mix the vector path (n % 8 == 0, one and several row chunks per
channel) with the element-wise path (n % 8 != 0), k = 0 matrices (m < 5 at
10%), and ragged channel counts.  tau = 0 ends every interval after one
step, tau = inf never triggers (the fixed schedule with S = S_max), and a
tau between observed ratios makes the trigger fire mid-interval.
"""
import math
import sys

import numpy as np
import pytest
import torch

import oracle as O
from tests._gpu import bits_np, f32_np, rel_close, same_bits
from workloads import base_scales, derive_seed, gradient, jittered_scales, space_boundary

pytestmark = pytest.mark.gpu

zf = pytest.importorskip("paper_2505_12242_amd")

SHAPES = [(264, 300), (4104, 70), (43, 77), (8192, 65), (16, 3), (128, 1000)]


def _inputs(shapes, ratio, T, seed, dev, layout=None, padded=False):
    """Device gradients per step and bf16 weights in `layout` (default
    channel-major), plus the logical host bit patterns the oracle takes.
    padded (row-major): gradient rows padded to 16 bytes, so that the plans
    run the 16-byte update."""
    cm = layout is None or layout == zf.CHANNEL_MAJOR
    slots, host = [], []
    for t in range(1, T + 1):
        dslot, hslot = [], []
        for q, (n, m) in enumerate(shapes):
            k = O.k_from_ratio(ratio, m)
            base = base_scales(m, 1.5, derive_seed(seed, q, "base"))
            s = space_boundary(jittered_scales(base, 0.05, derive_seed(seed, q, "jit", t)), k)
            g = gradient(n, m, s, derive_seed(seed, q, "grad", t), device=dev)
            hslot.append(bits_np(g))
            if cm:
                dslot.append(g.t().contiguous())
            elif padded:
                dslot.append(zf.alloc_stored(zf.ROW_MAJOR, n, m, torch.bfloat16, dev).copy_(g))
            else:
                dslot.append(g)
        slots.append(dslot)
        host.append(hslot)
    weights, w0 = [], []
    for q, (n, m) in enumerate(shapes):
        g = torch.Generator().manual_seed(derive_seed(seed, q, "w") & 0x7fffffff)
        w = (0.02 * torch.randn(n, m, generator=g)).to(torch.bfloat16)
        w0.append(bits_np(w))
        weights.append((w.t().contiguous() if cm else w).to(dev))
    return slots, host, weights, w0


def _oracle(shapes, w0, ratio, hp, R, S_max, tau):
    orcs = [O.MatrixOracle(O.widen(w0[q]), w0[q], ratio, hp.lr, hp.beta1, hp.beta2, hp.eps,
                           hp.weight_decay, R, S_max) for q in range(len(shapes))]
    return O.ZenAutoOracle(orcs, R, S_max, tau)


def _ratios(shapes, host, w0, ratio, hp, R, S_max):
    """(mean accumulated norm) / (mean selected norm) at every step of the
    fixed schedule (tau = inf), from the oracle."""
    za = _oracle(shapes, w0, ratio, hp, R, S_max, math.inf)
    out = []
    for grads in host:
        tot = za.step(grads)["totals"]
        out.append((tot.sum_acc / tot.u) / (tot.sum_sel / tot.k))
    return out


def _host(t, layout=None):
    if layout == zf.ROW_MAJOR:
        return t.contiguous().cpu()
    return t.t().contiguous().cpu()


def fixed_ends(T, R, S_max):
    """Interval ends when the trigger never fires: an interval starts at a
    refresh or after an end and ends at S_max steps or before a refresh."""
    ends, length, ended = [], 0, True
    for t in range(1, T + 1):
        length = 1 if ((t - 1) % R == 0 or ended) else length + 1
        ended = length >= S_max or t % R == 0
        ends.append(ended)
    return ends


def run_zen(shapes, ratio, R, S_max, tau, T, seed, host_in=None, layout=None, on_device=True,
            deferred=False):
    layout = zf.CHANNEL_MAJOR if layout is None else layout
    dev = torch.device("cuda")
    hp = zf.AdamHparams(lr=1e-3)
    slots, host, weights, w0 = host_in or _inputs(shapes, ratio, T, seed, dev, layout)
    runner = zf.SelectiveUpdateRunner(shapes, ratio, hp, R, S_max, slots, weights, device=dev,
                                      layout=layout, zen_tau=tau, zen_on_device=on_device,
                                      deferred_pack=deferred)
    # the interval decided on the device unless asked otherwise
    assert runner.zen_device == on_device
    za = _oracle(shapes, w0, ratio, hp, R, S_max, tau)
    ends = []
    exact_stats = total_stats = 0
    for t in range(1, T + 1):
        print(f"# zen-auto tau={tau} step {t}", file=sys.stderr, flush=True)
        kind = runner.step()
        torch.cuda.synchronize()
        ref = za.step(host[t - 1])
        assert (kind.refresh, kind.step_in_interval, kind.interval_end) == \
            (ref["refresh"], ref["step_in_interval"], ref["interval_end"]), t
        got, want = runner.last_totals, ref["totals"]
        assert (got.k_total, got.u_total) == (want.k, want.u)
        assert abs(got.sum_sel - want.sum_sel) <= 1e-9 * want.sum_sel, (t, got, want)
        assert abs(got.sum_acc - want.sum_acc) <= 1e-9 * want.sum_acc, (t, got, want)
        lhs = want.sum_acc * want.k
        rhs = tau * want.sum_sel * want.u
        if want.k and want.u and (math.isinf(tau) or abs(lhs - rhs) > 1e-9 * max(lhs, rhs)):
            assert got.trigger == want.trigger, (t, got, want)
        for q in range(len(shapes)):
            ssq, asq = ref["stats"][q]
            for dev_t, ref_v, name in ((runner.sel_sq[q], ssq, "sel_sq"),
                                       (runner.acc_sq[q], asq, "acc_sq")):
                g = f32_np(dev_t)
                ok, worst = rel_close(g, ref_v, 1e-5)
                assert ok, (name, q, t, worst)
                exact_stats += int(np.sum(g.view(np.uint32) == ref_v.view(np.uint32)))
                total_stats += g.size
            orc = za.orcs[q]
            P, M, V = (_host(x, layout).numpy() for x in runner.state[q])
            for a, b, name in ((P, orc.P, "master"), (M, orc.M, "exp_avg"),
                               (V, orc.V, "exp_avg_sq")):
                assert same_bits(a, b), (name, q, t)
            # (an end the caller forces is handed over by the update itself,
            # which leaves the packed buffer as it was; the hand-over below
            # carries the sums)
            # (deferred packing writes no packed buffer)
            if not deferred and not (kind.interval_end and getattr(kind, "fused", False)):
                assert same_bits(_host(runner.acc[q], layout).numpy(), orc.A), ("acc", q, t)
            wl = runner.weights[q] if layout == zf.ROW_MAJOR else runner.weights[q].t()
            assert same_bits(bits_np(wl), orc.W), ("weight", q, t)
            if kind.interval_end:
                assert same_bits(_host(runner.unpacked[q], layout).numpy(),
                                 ref["unpacked"][q]), ("hand-over", q, t)
        ends.append(kind.interval_end)
    runner.close()
    return ends, exact_stats, total_stats


LAYOUTS = [pytest.param(zf.ROW_MAJOR, id="rm"), pytest.param(zf.CHANNEL_MAJOR, id="cm")]
# the interval decided on the device (the default) and on the host
LAYOUT_MODES = [pytest.param(zf.ROW_MAJOR, True, False, id="rm-device"),
                pytest.param(zf.ROW_MAJOR, False, False, id="rm-host"),
                pytest.param(zf.CHANNEL_MAJOR, True, False, id="cm-device"),
                pytest.param(zf.CHANNEL_MAJOR, False, False, id="cm-host"),
                pytest.param(zf.CHANNEL_MAJOR, True, True, id="cm-device-deferred")]


@pytest.mark.timeout(600)
@pytest.mark.parametrize("tau", [0.0, math.inf])
@pytest.mark.parametrize("layout,on_device,deferred", LAYOUT_MODES)
def test_zen_auto_extreme_thresholds(tau, layout, on_device, deferred):
    T, R, S_max = 9, 4, 3
    ends, exact, total = run_zen(SHAPES, 0.1, R, S_max, tau, T, seed=11, layout=layout,
                                 on_device=on_device, deferred=deferred)
    if tau == 0.0:
        assert all(ends)
    else:
        # intervals of S_max steps, cut before each refresh (t = 5, 9)
        assert ends == fixed_ends(T, R, S_max) == [False, False, True, True, False, False,
                                                   True, True, False]
    print(f"# stats bit-exact: {exact}/{total}", file=sys.stderr, flush=True)


@pytest.mark.timeout(600)
@pytest.mark.parametrize("layout,on_device,deferred", LAYOUT_MODES)
def test_zen_auto_threshold_between_observed_ratios(layout, on_device, deferred):
    """tau between the ratios the fixed schedule produces after one and after
    several accumulated steps: the trigger fires mid-interval."""
    T, R, S_max, ratio = 10, 16, 6, 0.1
    dev = torch.device("cuda")
    inputs = _inputs(SHAPES, ratio, T, 12, dev, layout)
    r = _ratios(SHAPES, inputs[1], inputs[3], ratio, zf.AdamHparams(lr=1e-3), R, S_max)
    lo, hi = min(r[:2]), max(r[2:S_max])
    assert hi > lo
    tau = math.sqrt(lo * hi)
    ends, _, _ = run_zen(SHAPES, ratio, R, S_max, tau, T, seed=12, host_in=inputs, layout=layout,
                         on_device=on_device, deferred=deferred)
    assert any(ends) and not all(ends)
    # at least one interval ended by the trigger before reaching S_max
    lengths, cur = [], 0
    for e in ends:
        cur += 1
        if e:
            lengths.append(cur)
            cur = 0
    assert any(L < S_max for L in lengths), lengths


@pytest.mark.timeout(300)
@pytest.mark.parametrize("ratio", [0.0, 1.0])
@pytest.mark.parametrize("layout,deferred", [(zf.ROW_MAJOR, False), (zf.CHANNEL_MAJOR, False),
                                             (zf.CHANNEL_MAJOR, True)],
                         ids=["rm", "cm", "cm-deferred"])
def test_zen_auto_one_part_empty(ratio, layout, deferred):
    """k = 0 (nothing selected) or k = m (nothing accumulated): the trigger
    never fires and the schedule is the fixed one."""
    ends, _, _ = run_zen(SHAPES[:3], ratio, 4, 2, 0.0, 5, seed=13, layout=layout,
                         deferred=deferred)
    assert ends == fixed_ends(5, 4, 2) == [False, True, False, True, False]


@pytest.mark.timeout(300)
@pytest.mark.parametrize("layout", LAYOUTS)
def test_zen_auto_deterministic(layout):
    dev = torch.device("cuda")
    shapes = SHAPES[:4]
    slots, host, weights, w0 = _inputs(shapes, 0.1, 2, 14, dev, layout)
    outs = []
    for _ in range(2):
        ws = [w.clone() for w in weights]
        runner = zf.SelectiveUpdateRunner(shapes, 0.1, zf.AdamHparams(), 4, 4, slots, ws,
                                          device=dev, layout=layout, zen_tau=1.0)
        tots = []
        for _ in range(2):
            runner.step()
            tots.append(runner.zen_totals.cpu().numpy().tobytes())
        outs.append((tots, [f32_np(x).tobytes() for x in runner.acc_sq + runner.sel_sq]))
        runner.close()
    assert outs[0] == outs[1]


@pytest.mark.timeout(300)
@pytest.mark.parametrize("storage", ["cm", "cm-deferred", "rm", "rm-16B"])
@pytest.mark.parametrize("case", ["early-end", "warmup"])
def test_zen_auto_on_device_needs_no_host_round_trip(case, storage):
    """The device-decided interval: steps are enqueued without reading
    anything back (each returned step kind is unresolved until asked), and
    resolving them afterwards gives the host-decided run's positions, ends,
    hand-overs and states bit for bit -- with a threshold between the
    observed ratios (intervals ended by the trigger before S_max), and with
    a two-step warm-up.  Channel-major (packing every step, and deferred
    packing: the device run keeps the interval's gradients in their slots
    and sums them for the statistics), and row-major on the per-column
    update (unpadded rows) and on the 16-byte update (16-byte rows)."""
    dev = torch.device("cuda")
    layout = zf.CHANNEL_MAJOR if storage.startswith("cm") else zf.ROW_MAJOR
    padded = storage == "rm-16B"
    deferred = storage == "cm-deferred"
    if case == "early-end":
        T, R, S_max, warmup = 10, 16, 6, 0
        inputs = _inputs(SHAPES, 0.1, T, 12, dev, layout, padded)
        r = _ratios(SHAPES, inputs[1], inputs[3], 0.1, zf.AdamHparams(lr=1e-3), R, S_max)
        tau = math.sqrt(min(r[:2]) * max(r[2:S_max]))
    else:
        T, R, S_max, warmup, tau = 8, 4, 3, 2, 1.0
        inputs = _inputs(SHAPES, 0.1, T, 16, dev, layout, padded)
    results = []
    for on_device in (True, False):
        slots, _, weights, _ = inputs
        ws = [w.clone() for w in weights]
        runner = zf.SelectiveUpdateRunner(SHAPES, 0.1, zf.AdamHparams(lr=1e-3), R, S_max, slots,
                                          ws, device=dev, layout=layout, zen_tau=tau,
                                          warmup=warmup, zen_on_device=on_device,
                                          deferred_pack=deferred and on_device)
        assert runner.zen_device == on_device
        kinds, hand = [], []
        for t in range(T):
            kinds.append(runner.step())
            if on_device:
                assert kinds[-1]._vals is None  # nothing read back by the step
            hand.append([x.clone() for x in runner.unpacked])
        torch.cuda.synchronize()
        seq = [(k.refresh, k.step_in_interval, k.interval_end) for k in kinds]
        results.append((seq, [[f32_np(x) for x in h] for h, k in zip(hand, kinds)
                              if k.interval_end],
                        [f32_np(x) for q in range(len(SHAPES)) for x in runner.state[q]]))
        runner.close()
    (seq_d, hand_d, st_d), (seq_h, hand_h, st_h) = results
    assert seq_d == seq_h
    if case == "early-end":
        assert any(e and sii < S_max for _, sii, e in seq_d)
    else:
        assert all(e and sii == 1 for _, sii, e in seq_d[:warmup])
    assert len(hand_d) == len(hand_h)
    for a, b in zip(hand_d, hand_h):
        for x, y in zip(a, b):
            assert same_bits(x, y)
    for x, y in zip(st_d, st_h):
        assert same_bits(x, y)


def _plan_buffers(layout, with_stats=True):
    dev = torch.device("cuda")
    n, m = 64, 100
    k = O.k_from_ratio(0.1, m)
    shp = (lambda r, c: (r, c)) if layout == zf.ROW_MAJOR else (lambda r, c: (c, r))
    sel = zf.Selection(m, k, dev)
    f = dict(dtype=torch.float32, device=dev)
    return zf.MatrixBuffers(
        grad=torch.zeros(*shp(n, m), dtype=torch.bfloat16, device=dev), k=k, sel=sel,
        weight=torch.zeros(*shp(n, m), dtype=torch.bfloat16, device=dev),
        master=torch.zeros(*shp(n, k), **f), exp_avg=torch.zeros(*shp(n, k), **f),
        exp_avg_sq=torch.zeros(*shp(n, k), **f), acc=torch.zeros(*shp(n, m - k), **f),
        norms=torch.zeros(m, **f), layout=layout,
        sel_sq=torch.zeros(k, **f) if with_stats else None,
        acc_sq=torch.zeros(m - k, **f) if with_stats else None)


@pytest.mark.parametrize("layout,with_stats", [(0, False), (1, False)])
def test_zen_auto_rejected_without_statistics_buffers(layout, with_stats):
    """Plans without statistics buffers refuse the call (ZF_EINVAL) and
    enqueue nothing."""
    plan = zf.Plan([_plan_buffers(layout, with_stats)])
    plan.colnorm()
    plan.topk_select()  # a valid selection, should anything run
    totals = torch.zeros(5, dtype=torch.int64, device="cuda")
    with pytest.raises(zf.ZfError, match="invalid argument"):
        plan.update_zen(zf.AdamHparams(), 1, zf.STATES_INIT, 1, 4, 1.0, totals)
    torch.cuda.synchronize()
    assert not totals.any()
    plan.close()


def test_zen_auto_rejects_bad_arguments():
    plan = zf.Plan([_plan_buffers(zf.CHANNEL_MAJOR)])
    plan.colnorm()
    plan.topk_select()  # zero gradient: the first k channels
    totals = torch.zeros(5, dtype=torch.int64, device="cuda")
    hp = zf.AdamHparams()
    for args in ((hp, 1, zf.STATES_INIT, 1, 4, float("nan")),
                 (hp, 1, zf.STATES_INIT, 1, 4, -1.0),
                 (hp, 0, zf.STATES_INIT, 1, 4, 1.0),
                 (hp, 1, zf.STATES_INIT, 5, 4, 1.0)):
        with pytest.raises(zf.ZfError):
            plan.update_zen(*args, totals)
    plan.update_zen(hp, 1, zf.STATES_INIT, 1, 4, 1.0, totals)
    torch.cuda.synchronize()
    tot = zf.ZenTotals.from_bytes(totals.cpu().numpy().tobytes())
    assert (tot.k_total, tot.u_total) == (10, 90)
    assert tot.sum_sel == 0.0 and tot.sum_acc == 0.0 and tot.trigger  # 0 >= tau * 0
    plan.close()


def test_zen_deferred_rejects_bad_arguments():
    """zf_plan_update_zen_deferred / zf_plan_handover_zen_deferred validate on
    the host, with nothing enqueued: a plan without `unpacked` or a row-major
    plan, more than 15 earlier plans, an earlier plan over other matrices, a
    bad force_end or tau, a missing state."""
    dev = torch.device("cuda")
    totals = torch.zeros(5, dtype=torch.int64, device=dev)
    state = torch.tensor([0, 1], dtype=torch.int32, device=dev)
    hp = zf.AdamHparams()

    def with_out(layout):
        b = _plan_buffers(layout)
        n, m = 64, 100
        b.unpacked = torch.zeros(*((n, m) if layout == zf.ROW_MAJOR else (m, n)),
                                 dtype=torch.float32, device=dev)
        return b

    plan = zf.Plan([with_out(zf.CHANNEL_MAJOR)])
    other = zf.Plan([with_out(zf.CHANNEL_MAJOR), with_out(zf.CHANNEL_MAJOR)])
    rm = zf.Plan([with_out(zf.ROW_MAJOR)])
    no_out = zf.Plan([_plan_buffers(zf.CHANNEL_MAJOR)])
    before = state.clone()
    bad = [
        (rm, [], 2, 1.0, state),              # row-major
        (no_out, [], 2, 1.0, state),          # no hand-over buffer
        (plan, [plan] * 16, 2, 1.0, state),   # more than 15 earlier plans
        (plan, [other], 2, 1.0, state),       # other matrices
        (plan, [], 3, 1.0, state),            # force_end
        (plan, [], 2, -1.0, state),           # tau
    ]
    for pl, earlier, fe, tau, st in bad:
        with pytest.raises(zf.ZfError, match="invalid argument"):
            pl.update_zen_deferred(hp, 1, zf.STATES_INIT, 4, earlier, fe, tau, totals, st)
    for pl, earlier in ((rm, []), (no_out, []), (plan, [plan] * 16), (plan, [other])):
        with pytest.raises(zf.ZfError, match="invalid argument"):
            pl.handover_zen_deferred(earlier, state)
    torch.cuda.synchronize()
    assert torch.equal(state, before)
    for pl in (plan, other, rm, no_out):
        pl.close()


def test_rowmajor_fused_statistics_equal_separate_pass():
    """Row-major plans: the statistics fused into the 16-byte update (aligned,
    padded buffers) and the separate statistics pass (the same data in
    unaligned buffers, per-column update) write the same partials: the
    per-channel statistics, the totals, the states and the packed buffer are
    equal bit for bit, over an init step and two in-place steps."""
    from tests._gpu import bf16_dev, bits_np
    from workloads import derive_seed, gradient
    shapes = [(40, 1009), (17, 77), (64, 2048)]
    hp = zf.AdamHparams(lr=1e-3)
    rng = np.random.default_rng(23)

    def f32(a, aligned):
        n, w = a.shape
        if aligned:
            t = zf.alloc_stored(zf.ROW_MAJOR, n, w)
        else:
            t = torch.empty(n * w + 1, device="cuda")[1:].view(n, w)
        t.copy_(torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)))
        return t

    def bf16(bits, aligned):
        m = bits.shape[1]
        return bf16_dev(bits, ld=-(-m // 8) * 8) if aligned else bf16_dev(bits, offset=1)

    grads = {}
    sets = {True: [], False: []}
    sels = []
    for q, (n, m) in enumerate(shapes):
        k = zf.k_from_ratio(0.1, m)
        sel = O.select_topk(rng.random(m).astype(np.float32), k)
        s = zf.Selection(m, k)
        s.sel_idx.copy_(torch.from_numpy(sel.sel.astype(np.int32)))
        s.unsel_idx.copy_(torch.from_numpy(sel.unsel.astype(np.int32)))
        s.mask.copy_(torch.from_numpy(sel.mask.view(np.int64)))
        s.prefix.copy_(torch.from_numpy(sel.prefix.astype(np.int32)))
        sels.append(s)
        W = O.bf16_round((rng.standard_normal((n, m)) * 0.02).astype(np.float32))
        for t in (1, 2, 3):
            g = torch.Generator().manual_seed(derive_seed("zen-fused", q, t))
            sc = torch.exp(1.5 * torch.randn(m, generator=g, dtype=torch.float64))
            grads[q, t] = bits_np(gradient(n, m, sc, seed=derive_seed("zen-fused", q, t)))
        for al in (True, False):
            sets[al].append(dict(
                G=[bf16(grads[q, t], al) for t in (1, 2, 3)], W=bf16(W, al),
                P=f32(np.zeros((n, k)), al), M=f32(np.zeros((n, k)), al),
                V=f32(np.zeros((n, k)), al), A=f32(np.zeros((n, m - k)), al),
                ssq=torch.empty(k, device="cuda"), asq=torch.empty(m - k, device="cuda")))
    results = {}
    for al in (True, False):
        totals_seq = []
        for t in (1, 2, 3):
            mats = [zf.MatrixBuffers(grad=b["G"][t - 1], k=sels[q].k, sel=sels[q], weight=b["W"],
                                     master=b["P"], exp_avg=b["M"], exp_avg_sq=b["V"], acc=b["A"],
                                     layout=zf.ROW_MAJOR, sel_sq=b["ssq"], acc_sq=b["asq"])
                    for q, b in enumerate(sets[al])]
            plan = zf.Plan(mats)
            totals = torch.zeros(5, dtype=torch.int64, device="cuda")
            plan.update_zen(hp, t, zf.STATES_INIT if t == 1 else zf.STATES_INPLACE, t, 4,
                            math.inf, totals)
            torch.cuda.synchronize()
            totals_seq.append(totals.cpu().numpy().tobytes())
            plan.close()
        results[al] = (totals_seq, [[x.cpu().numpy().tobytes() for x in
                                     (b["ssq"], b["asq"], b["P"].contiguous(), b["M"].contiguous(),
                                      b["V"].contiguous(), b["A"].contiguous())]
                                    for b in sets[al]])
    assert results[True][0] == results[False][0]
    assert results[True][1] == results[False][1]
