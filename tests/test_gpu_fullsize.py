"""Parity at full size, in the launch configuration bench.py times (batched
plans, three-slot gradient ring): the whole Llama-2-7B-shaped gradient set
(226 matrices) for 8 steps of the R = S = 4 schedule -- first selection,
accumulation, hand-over at step 4, refresh with state remap at step 5,
hand-over at step 8 -- in both layouts (channel-major, bench.py's default,
and row-major with the 16-byte update), and one R = S = 8 interval of the
70B share (heavy-tailed scales, GQA k/v weights, 28672-channel down
projections) in the channel-major layout.  Both packing modes run: every
step (packed sums updated by each step) and deferred (bench.py's default:
the interval's gradients stay in a ring of min(S, R) slots and its last
step sums them), the 7B set in both layouts.

* Sampled matrices (embedding, LM head and four decoder weights of three
  shapes) are run through the oracle step by step and every output is
  compared in full.
* Every matrix is checked for properties that hold at any size: the
  selection is a partition of size k that ranks the scores the kernels
  produced, and the scores sum to the squared Frobenius norm of the
  gradient computed by torch in fp64.
"""
import sys

import numpy as np
import pytest
import torch

import oracle as O
from tests._gpu import bits_np, f32_np, mask_np, rel_close, same_bits

pytestmark = pytest.mark.gpu

zf = pytest.importorskip("paper_2505_12242_amd")
bench = pytest.importorskip("bench")

CASES = {
    # first selection, accumulation, hand-over at 4, refresh + remap at 5, hand-over at 8
    "llama2-7b-full": (["embed_tokens", "layers.0.q_proj", "layers.0.down_proj",
                        "layers.17.gate_proj", "layers.31.v_proj", "lm_head"], 8, 3, []),
    # one R = S = 8 interval of the 70B share: heavy-tailed scales, the GQA k/v
    # weight (1024 rows) against the oracle in full, and a 28672-channel down
    # projection through cheaper checks (its selection against the oracle's
    # top-k of the device scores; its hand-over recomputed on the device in
    # the kernels' fp32 order)
    "llama2-70b-10layers": (["layers.0.k_proj"], 8, 3, ["layers.9.down_proj"]),
}


RUNS = [("llama2-7b-full", "cm"), ("llama2-7b-full", "cm-deferred"), ("llama2-7b-full", "rm"),
        ("llama2-7b-full", "rm-deferred"), ("llama2-70b-10layers", "cm"),
        ("llama2-70b-10layers", "cm-deferred")]
# the row-major run compares the three decoder shapes in full (the 32000-row
# embedding and head, the slowest oracle work, are compared in the
# channel-major run; every matrix gets the property checks in both)
RM_SAMPLES = ["layers.0.q_proj", "layers.0.down_proj", "layers.17.gate_proj"]


def logical_cm(t):
    """Logical [out, in] view of a channel-major tensor."""
    return t.t()


@pytest.mark.timeout(1200)
@pytest.mark.parametrize("name,lay", RUNS)
def test_full_set_sampled_parity(name, lay):
    from workloads import get_workload
    SAMPLES, STEPS, NSLOTS, LIGHT = CASES[name]
    if lay.startswith("rm"):
        SAMPLES = RM_SAMPLES
    deferred = lay.endswith("-deferred")  # bench.py's default packing: the interval in the ring
    wl = get_workload(name)
    if deferred:
        NSLOTS = min(wl.accum, wl.refresh)
    hp = zf.AdamHparams(wl.hyper.lr, wl.hyper.beta1, wl.hyper.beta2, wl.hyper.eps,
                        wl.hyper.weight_decay)
    dev = torch.device("cuda")
    layout = zf.ROW_MAJOR if lay.startswith("rm") else zf.CHANNEL_MAJOR
    assert not LIGHT or layout == zf.CHANNEL_MAJOR  # the light checks index channel rows

    def logical(t):
        return t.t() if layout == zf.CHANNEL_MAJOR else t
    shapes, ks, slots, weights = bench.build_set(wl, NSLOTS, dev, layout)
    names = [mt.name for mt in wl.matrices]
    qs = [names.index(s) for s in SAMPLES]
    light = [names.index(s) for s in LIGHT]
    w0 = {q: bits_np(logical(weights[q]).contiguous()) for q in qs}
    g_host = {(q, s): bits_np(logical(slots[s][q]).contiguous()) for q in qs
              for s in range(NSLOTS)}
    runner = zf.SelectiveUpdateRunner(shapes, wl.ratio, hp, wl.refresh, wl.accum, slots, weights,
                                      device=dev, layout=layout, deferred_pack=deferred)
    orcs = {q: O.MatrixOracle(O.widen(w0[q]), w0[q], wl.ratio, hp.lr, hp.beta1, hp.beta2,
                              hp.eps, hp.weight_decay, wl.refresh, wl.accum) for q in qs}
    for t in range(1, STEPS + 1):
        kind = runner.step()
        torch.cuda.synchronize()
        slot = (t - 1) % NSLOTS
        print(f"# step {t} ({'refresh' if kind.refresh else 'accumulate'})", file=sys.stderr,
              flush=True)
        for q in light:
            if kind.refresh:
                # exact top-k of the device's own scores
                want = O.select_topk(f32_np(runner.norms[q]), ks[q])
                got = runner.selection[q]
                assert np.array_equal(got.sel_idx.cpu().numpy(), want.sel), (names[q], t)
                assert np.array_equal(mask_np(got.mask), want.mask), (names[q], t)
            if kind.interval_end:
                # hand-over = fp32(1/length) * (((g_1 + g_2) + ...) + g_t) at the
                # unselected channels, +0.0 at the selected ones (channel rows)
                unsel = runner.selection[q].unsel_idx.long()
                start = t - kind.step_in_interval + 1
                acc = slots[(start - 1) % NSLOTS][q].float()[unsel]
                for tt in range(start + 1, t + 1):
                    acc = acc + slots[(tt - 1) % NSLOTS][q].float()[unsel]
                want = torch.zeros_like(runner.unpacked[q])
                want[unsel] = acc * torch.tensor(np.float32(1.0 / kind.step_in_interval),
                                                 device=acc.device)
                assert torch.equal(runner.unpacked[q].view(torch.int32),
                                   want.view(torch.int32)), (names[q], t)
        if kind.refresh:
            for q, (n, m) in enumerate(shapes):
                s = f32_np(runner.norms[q]).astype(np.float64)
                sel = runner.selection[q]
                a = sel.sel_idx.cpu().numpy()
                b = sel.unsel_idx.cpu().numpy()
                assert a.size == ks[q] and b.size == m - ks[q]
                assert np.array_equal(np.sort(np.concatenate([a, b])), np.arange(m))
                assert s[a].min() >= s[b].max(), names[q]
                frob = torch.sum(slots[slot][q].double() ** 2).item()
                assert abs(s.sum() - frob) <= 1e-6 * frob, names[q]
        for q in qs:
            out = orcs[q].step(g_host[(q, slot)])
            orc = orcs[q]
            nm = names[q]
            if kind.refresh:
                ok, worst = rel_close(f32_np(runner.norms[q]), out["norms"], 1e-5)
                assert ok, (nm, t, worst)
                sel = runner.selection[q]
                assert np.array_equal(sel.sel_idx.cpu().numpy(), orc.sel.sel), (nm, t)
                assert np.array_equal(sel.unsel_idx.cpu().numpy(), orc.sel.unsel), (nm, t)
                assert np.array_equal(mask_np(sel.mask), orc.sel.mask), (nm, t)
                assert np.array_equal(sel.prefix.cpu().numpy(), orc.sel.prefix), (nm, t)
            P, M, V = (f32_np(logical(x)) for x in runner.state[q])
            assert same_bits(P, orc.P) and same_bits(M, orc.M) and same_bits(V, orc.V), (nm, t)
            # the packed buffer after the overwrite and the first accumulation
            # (the interval's last step hands over without writing it; the
            # hand-over is compared below)
            if kind.step_in_interval <= 2 and not kind.interval_end and not deferred:
                assert same_bits(f32_np(logical(runner.acc[q])), orc.A), (nm, t)
            assert np.array_equal(bits_np(logical(weights[q]).contiguous()), orc.W), (nm, t)
            if kind.interval_end:
                assert same_bits(f32_np(logical(runner.unpacked[q])), out["unpacked"]), (nm, t)
    runner.close()
    del runner, slots, weights
    torch.cuda.empty_cache()


@pytest.mark.timeout(900)
def test_full_set_zen_auto_statistics():
    """Zen-auto over the whole 7B set in bench.py's launch configuration
    (channel-major, batched, three-slot ring), 3 steps with tau = inf (the
    fixed schedule): the device totals equal fp64 sums, recomputed on the
    host, of the device's own per-channel statistics (all 1.15 M channels),
    k and u totals are exact, and two sampled matrices' statistics match the
    oracle within 1e-5 (their states and packed buffers bit for bit)."""
    import math
    from workloads import get_workload
    wl = get_workload("llama2-7b-full")
    hp = zf.AdamHparams(wl.hyper.lr, wl.hyper.beta1, wl.hyper.beta2, wl.hyper.eps,
                        wl.hyper.weight_decay)
    dev = torch.device("cuda")
    shapes, ks, slots, weights = bench.build_set(wl, 3, dev, zf.CHANNEL_MAJOR)
    names = [mt.name for mt in wl.matrices]
    qs = [names.index("layers.5.up_proj"), names.index("lm_head")]
    w0 = {q: bits_np(logical_cm(weights[q]).contiguous()) for q in qs}
    runner = zf.SelectiveUpdateRunner(shapes, wl.ratio, hp, wl.refresh, wl.accum, slots, weights,
                                      device=dev, layout=zf.CHANNEL_MAJOR, zen_tau=math.inf)
    orcs = {q: O.MatrixOracle(O.widen(w0[q]), w0[q], wl.ratio, hp.lr, hp.beta1, hp.beta2,
                              hp.eps, hp.weight_decay, wl.refresh, wl.accum) for q in qs}
    for t in range(1, 4):
        kind = runner.step()
        torch.cuda.synchronize()
        print(f"# zen full set step {t}", file=sys.stderr, flush=True)
        tot = runner.last_totals
        assert tot.k_total == sum(ks) and tot.u_total == sum(m - k for (_, m), k in zip(shapes, ks))
        assert not tot.trigger
        sel_all = torch.cat(runner.sel_sq).double()
        acc_all = torch.cat(runner.acc_sq).double()
        assert abs(torch.sqrt(sel_all).sum().item() - tot.sum_sel) <= 1e-9 * tot.sum_sel
        assert abs(torch.sqrt(acc_all).sum().item() - tot.sum_acc) <= 1e-9 * tot.sum_acc
        for q in qs:
            G = bits_np(logical_cm(slots[(t - 1) % 3][q]).contiguous())
            orcs[q].advance(G, kind.refresh, kind.step_in_interval)
            ssq, asq = O.zen_auto_stats(G, orcs[q].sel, orcs[q].A)
            ok, worst = rel_close(f32_np(runner.sel_sq[q]), ssq, 1e-5)
            assert ok, (names[q], t, worst)
            ok, worst = rel_close(f32_np(runner.acc_sq[q]), asq, 1e-5)
            assert ok, (names[q], t, worst)
            assert same_bits(f32_np(logical_cm(runner.acc[q])), orcs[q].A), (names[q], t)
            P = f32_np(logical_cm(runner.state[q][0]))
            assert same_bits(P, orcs[q].P), (names[q], t)
    runner.close()
    del runner, slots, weights
    torch.cuda.empty_cache()


@pytest.mark.timeout(900)
@pytest.mark.parametrize("lay", ["cm", "rm"])
def test_full_set_deferred_equals_every_step_over_48_steps(lay):
    """The whole 7B set for 48 steps of the R = S = 4 schedule (12
    refreshes, 12 interval ends), once with deferred packing (bench.py's
    default) and once packing every step: every matrix's W, compact states,
    selection and final hand-over are equal bit for bit (torch.equal on the
    device, all 226 matrices)."""
    from workloads import get_workload
    wl = get_workload("llama2-7b-full")
    hp = zf.AdamHparams(wl.hyper.lr, wl.hyper.beta1, wl.hyper.beta2, wl.hyper.eps,
                        wl.hyper.weight_decay)
    dev = torch.device("cuda")
    layout = zf.ROW_MAJOR if lay == "rm" else zf.CHANNEL_MAJOR
    steps, nslots = 48, 4
    kept = None
    for deferred in (True, False):
        torch.cuda.empty_cache()
        shapes, ks, slots, weights = bench.build_set(wl, nslots, dev, layout)
        runner = zf.SelectiveUpdateRunner(shapes, wl.ratio, hp, wl.refresh, wl.accum, slots,
                                          weights, device=dev, layout=layout,
                                          deferred_pack=deferred)
        for t in range(1, steps + 1):
            kind = runner.step()
        torch.cuda.synchronize()
        assert kind.interval_end
        print(f"# {lay} deferred={deferred}: {steps} steps done", file=sys.stderr, flush=True)
        out = [(weights[q], *runner.state[q], runner.unpacked[q],
                runner.selection[q].sel_idx) for q in range(len(shapes))]
        if kept is None:
            kept = [tuple(x.clone() for x in o) for o in out]
        else:
            bits = {torch.float32: torch.int32, torch.bfloat16: torch.int16}
            for q, (a, b) in enumerate(zip(kept, out)):
                for x, y in zip(a, b):
                    assert torch.equal(x.view(bits.get(x.dtype, x.dtype)),
                                       y.view(bits.get(y.dtype, y.dtype))), q
        runner.close()
        del runner, slots, weights, out
    del kept
    torch.cuda.empty_cache()


@pytest.mark.timeout(900)
def test_full_set_zen_deferred_equals_every_step():
    """Zen-auto over the whole 7B set in bench.py's launch configuration for
    it (channel-major, decided on the device, tau = 1, R = S = 4, a four-slot
    ring), 16 steps, once with deferred packing (bench.py's default there)
    and once packing every step: the same interval positions and ends and
    the same 40-byte totals at every step, and at the end every matrix's W,
    compact states, selection and hand-over equal bit for bit (torch.equal
    on the device, all 226 matrices)."""
    from workloads import get_workload
    wl = get_workload("llama2-7b-full")
    hp = zf.AdamHparams(wl.hyper.lr, wl.hyper.beta1, wl.hyper.beta2, wl.hyper.eps,
                        wl.hyper.weight_decay)
    dev = torch.device("cuda")
    steps, nslots = 16, 4
    kept = None
    for deferred in (True, False):
        torch.cuda.empty_cache()
        shapes, ks, slots, weights = bench.build_set(wl, nslots, dev, zf.CHANNEL_MAJOR)
        runner = zf.SelectiveUpdateRunner(shapes, wl.ratio, hp, wl.refresh, wl.accum, slots,
                                          weights, device=dev, layout=zf.CHANNEL_MAJOR,
                                          zen_tau=1.0, deferred_pack=deferred)
        assert runner.zen_device and runner.deferred == deferred
        seq = []
        for t in range(1, steps + 1):
            kind = runner.step()
            tot = runner.last_totals  # resolves the step (a read-back after it)
            seq.append((kind.refresh, kind.step_in_interval, kind.interval_end,
                        tot.k_total, tot.u_total, tot.sum_sel, tot.sum_acc, tot.trigger))
        torch.cuda.synchronize()
        assert seq[-1][2]  # the last step ends an interval (a refresh follows)
        print(f"# zen full set deferred={deferred}: {steps} steps, ends at "
              f"{[t + 1 for t, s in enumerate(seq) if s[2]]}", file=sys.stderr, flush=True)
        out = [(weights[q], *runner.state[q], runner.unpacked[q],
                runner.selection[q].sel_idx) for q in range(len(shapes))]
        if kept is None:
            kept = (seq, [tuple(x.clone() for x in o) for o in out])
        else:
            assert seq == kept[0]
            bits = {torch.float32: torch.int32, torch.bfloat16: torch.int16}
            for q, (a, b) in enumerate(zip(kept[1], out)):
                for x, y in zip(a, b):
                    assert torch.equal(x.view(bits.get(x.dtype, x.dtype)),
                                       y.view(bits.get(y.dtype, y.dtype))), q
        runner.close()
        del runner, slots, weights, out
    del kept
    torch.cuda.empty_cache()
