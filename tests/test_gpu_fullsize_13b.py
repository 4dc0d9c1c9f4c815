"""Parity at the Llama-2-13B shapes (hidden 5120, FFN 13824, vocab 32000):
the paper's 13B model (Evaluation, Table "Experimental environments") and
its sweep of the top-k ratio and the selection refresh interval
(Evaluation, "Sensitivity of Hyperparameters"), in bench.py's launch
configuration: batched plans over the whole set, a ring of gradient slots,
the channel-major layout, and the hand-over fused into each interval's last
update (one-step intervals take it from the score pass).

* test_13b_full_set: all 282 matrices (13.0 G parameters) for 8 steps of
  the R = S = 4 schedule at ratio 10% -- first selection, accumulation,
  hand-over at 4, refresh with state remap at 5, hand-over at 8 -- in both
  packing modes: deferred (bench.py's default: the interval's gradients
  stay in a four-slot ring and its last step sums them,
  zf_plan_update_handover_deferred) and every step (the bf16 stage, then
  fp32 packed sums).
* test_13b_sweep: the 13B shapes (embedding, one decoder layer: 5120^2,
  13824 x 5120, 5120 x 13824, LM head) at ratios 1%, 5% and 25% with R = 1
  (every step refreshes and hands over at once: zf_plan_colnorm_handover,
  then zf_plan_update_adam_handover) and R = 16 (four S = 4 intervals with
  deferred packing, then a refresh with state remap), S = 4.

Checks, every matrix, every step:
* on refresh steps the selection (indices, mask, prefix) is the exact
  top-k of the scores the device produced, the scores sum to the squared
  Frobenius norm of the gradient (fp64, torch), and the scores of sampled
  columns (the k-th and (k+1)-th ranked among them) match the oracle's
  colnorm within 1e-5 (scores are per column, so a column subset is exact);
* sampled rows of every output -- compact states P/M/V, the bf16 weight,
  the packed sums (or the bf16 stage after an interval's first step; with
  deferred packing there are none) and the hand-over -- equal, bit for bit, the oracle's composition run on those
  rows under the device's selection (every step but the scores is
  row-wise, so the rows of the outputs follow from the rows of the inputs).
Sampled matrices are in addition run through the oracle in full
(MatrixOracle, its own scores and selection) and every output compared:
scores within 1e-5, everything else bit for bit.
"""
import sys
from concurrent.futures import ThreadPoolExecutor

import numpy as np
import pytest
import torch

import oracle as O
from tests._gpu import bits_np, f32_np, mask_np, rel_close, same_bits

pytestmark = pytest.mark.gpu

zf = pytest.importorskip("paper_2505_12242_amd")
bench = pytest.importorskip("bench")


def sample_rows(n, seed):
    """Row sample: ends, middle, the update kernel's row-chunk boundaries,
    and random rows."""
    rows = {0, 1, n // 2, n - 1}
    rows |= {b for c in (2048, 4096) for j in range(1, 8) for b in (j * c - 1, j * c) if b < n}
    rng = np.random.default_rng(seed)
    rows |= set(rng.integers(0, n, size=10).tolist())
    return torch.tensor(sorted(rows), dtype=torch.long)


def host_selection(s) -> O.Selection:
    return O.Selection(s.sel_idx.cpu().numpy().astype(np.int32),
                       s.unsel_idx.cpu().numpy().astype(np.int32),
                       mask_np(s.mask).copy(), s.prefix.cpu().numpy().astype(np.int32), s.m)


def rows_of(t, rows):
    """Logical [len(rows), width] rows of a channel-major [width, n] tensor."""
    x = t.index_select(1, rows.to(t.device))
    if x.dtype == torch.bfloat16:
        return np.ascontiguousarray(bits_np(x).T)
    return np.ascontiguousarray(f32_np(x).T)


class RowReplay:
    """The oracle's per-step composition (MatrixOracle.advance / hand_over)
    restricted to a subset of a matrix's rows, under a given selection."""

    def __init__(self, w_rows, hyper):
        self.W = np.array(w_rows, np.uint16, copy=True)
        self.master = O.widen(self.W)
        self.hyper = hyper
        self.t = 0
        self.sel = None
        self.P = self.M = self.V = self.A = None

    def advance(self, g_rows, sel, refresh, sii):
        self.t += 1
        if refresh:
            first = self.sel is None
            self.P, self.M, self.V = O.remap(self.sel, sel, self.P, self.M, self.V, self.W,
                                             self.master if first else None)
            self.sel = sel
        c = O.AdamConsts.at_step(*self.hyper, self.t)
        self.P, self.M, self.V, wsel = O.adam_selected(g_rows, self.sel.sel, self.P, self.M,
                                                       self.V, c)
        self.W[:, self.sel.sel.astype(np.int64)] = wsel
        self.A = O.pack_accumulate(g_rows, self.sel.unsel, self.A, sii)

    def hand_over(self, steps):
        return O.unpack(self.A, self.sel, float(np.float32(1.0 / steps)))


def run_and_check(wl, nslots, steps, full_names, tag, deferred=False):
    hp = zf.AdamHparams(wl.hyper.lr, wl.hyper.beta1, wl.hyper.beta2, wl.hyper.eps,
                        wl.hyper.weight_decay)
    hyper = (hp.lr, hp.beta1, hp.beta2, hp.eps, hp.weight_decay)
    dev = torch.device("cuda")
    torch.cuda.empty_cache()
    layout = zf.CHANNEL_MAJOR
    shapes, ks, slots, weights = bench.build_set(wl, nslots, dev, layout)
    names = [mt.name for mt in wl.matrices]
    full = [names.index(s) for s in full_names]
    rows = [sample_rows(n, q) for q, (n, m) in enumerate(shapes)]
    replay = [RowReplay(rows_of(weights[q], rows[q]), hyper) for q in range(len(shapes))]
    w0 = {q: bits_np(weights[q].t().contiguous()) for q in full}
    orcs = {q: O.MatrixOracle(O.widen(w0[q]), w0[q], wl.ratio, *hyper, wl.refresh, wl.accum)
            for q in full}
    del w0
    runner = zf.SelectiveUpdateRunner(shapes, wl.ratio, hp, wl.refresh, wl.accum, slots, weights,
                                      device=dev, layout=layout, deferred_pack=deferred)
    assert runner.fuse_handover and runner.use_stage != deferred
    pool = ThreadPoolExecutor(max(1, len(full)))
    try:
        for t in range(1, steps + 1):
            kind = runner.step()
            torch.cuda.synchronize()
            slot = (t - 1) % nslots
            sii, end = kind.step_in_interval, kind.interval_end
            print(f"# {tag} step {t}: refresh={kind.refresh} step_in_interval={sii} end={end}",
                  file=sys.stderr, flush=True)
            # the full oracle of the sampled matrices runs beside the checks below
            g_full = {q: bits_np(slots[slot][q].t().contiguous()) for q in full}
            futs = {q: pool.submit(orcs[q].step, g_full[q]) for q in full}
            col_checks = {}  # n -> [(q, sampled columns, device scores, gradient columns)]
            for q, (n, m) in enumerate(shapes):
                sel = runner.selection[q]
                if kind.refresh:
                    s = f32_np(runner.norms[q])
                    want = O.select_topk(s, ks[q])
                    assert np.array_equal(sel.sel_idx.cpu().numpy(), want.sel), (names[q], t)
                    assert np.array_equal(sel.unsel_idx.cpu().numpy(), want.unsel), (names[q], t)
                    assert np.array_equal(mask_np(sel.mask), want.mask), (names[q], t)
                    assert np.array_equal(sel.prefix.cpu().numpy(), want.prefix), (names[q], t)
                    frob = torch.sum(slots[slot][q].double() ** 2).item()
                    assert abs(s.astype(np.float64).sum() - frob) <= 1e-6 * frob, names[q]
                    # sampled columns for the oracle's colnorm: the boundary pair
                    # of the ranking and a few others
                    order = np.lexsort((np.arange(m), -s.astype(np.float64)))
                    cols = {int(order[min(ks[q], m - 1)]), int(order[max(ks[q] - 1, 0)]),
                            0, m - 1}
                    cols = np.array(sorted(cols | set(
                        np.random.default_rng(t * 7919 + q).integers(0, m, 6).tolist())))
                    g_cols = bits_np(slots[slot][q].index_select(
                        0, torch.from_numpy(cols).to(dev)).t().contiguous())
                    col_checks.setdefault(n, []).append((q, cols, s[cols], g_cols))
                # sampled rows of every output against the row-wise oracle composition
                r = rows[q]
                rp = replay[q]
                rp.advance(rows_of(slots[slot][q], r), host_selection(sel) if kind.refresh
                           else rp.sel, kind.refresh, sii)
                P, M, V = (rows_of(x, r) for x in runner.state[q])
                assert same_bits(P, rp.P) and same_bits(M, rp.M) and same_bits(V, rp.V), \
                    (names[q], t)
                assert np.array_equal(rows_of(weights[q], r), rp.W), (names[q], t)
                if end:
                    assert same_bits(rows_of(runner.unpacked[q], r), rp.hand_over(sii)), \
                        (names[q], t)
                elif not deferred:  # deferred packing keeps no sums between steps
                    if runner._in_stage:
                        stage_rows = runner.stage[q].index_select(1, r.to(dev))
                        a = O.widen(np.ascontiguousarray(bits_np(
                            stage_rows.index_select(0, sel.unsel_idx.long())).T))
                    else:
                        a = rows_of(runner.current_acc[q], r)
                    assert same_bits(a, rp.A), (names[q], t)
            # scores are per column: one oracle colnorm over the sampled
            # columns of all matrices with the same row count
            for n, items in col_checks.items():
                want = O.colnorm(np.concatenate([g for *_, g in items], axis=1))
                at = 0
                for q, cols, got, _ in items:
                    ok, worst = rel_close(got, want[at: at + cols.size], 1e-5)
                    assert ok, (names[q], t, worst)
                    at += cols.size
            for q in full:
                out = futs[q].result()
                orc = orcs[q]
                nm = names[q]
                sel = runner.selection[q]
                if kind.refresh:
                    ok, worst = rel_close(f32_np(runner.norms[q]), out["norms"], 1e-5)
                    assert ok, (nm, t, worst)
                    assert np.array_equal(sel.sel_idx.cpu().numpy(), orc.sel.sel), (nm, t)
                    assert np.array_equal(mask_np(sel.mask), orc.sel.mask), (nm, t)
                P, M, V = (f32_np(x.t()) for x in runner.state[q])
                assert same_bits(P, orc.P) and same_bits(M, orc.M) and same_bits(V, orc.V), \
                    (nm, t)
                assert np.array_equal(bits_np(weights[q].t().contiguous()), orc.W), (nm, t)
                if end:
                    assert same_bits(f32_np(runner.unpacked[q].t()), out["unpacked"]), (nm, t)
            del g_full, futs
    finally:
        pool.shutdown(wait=True)
        runner.close()
        del runner, slots, weights
        torch.cuda.empty_cache()


@pytest.mark.timeout(1200)
@pytest.mark.parametrize("packing", ["deferred", "every-step"])
def test_13b_full_set(packing):
    from workloads import get_workload
    wl = get_workload("llama2-13b-full")
    assert len(wl.matrices) == 282 and wl.params == 13_015_449_600
    deferred = packing == "deferred"
    # deferred packing keeps the interval's S = 4 gradients in the ring
    run_and_check(wl, 4 if deferred else 2, 8,
                  ["layers.0.q_proj", "layers.0.gate_proj", "layers.39.down_proj", "lm_head"],
                  f"13b-full {packing}", deferred=deferred)


SWEEP = [(0.01, 1, 3, "layers.0.gate_proj"), (0.05, 1, 3, "layers.0.down_proj"),
         (0.25, 1, 3, "layers.0.q_proj"),
         (0.01, 16, 17, "layers.0.q_proj"), (0.05, 16, 17, "layers.0.q_proj"),
         (0.25, 16, 17, "layers.0.q_proj")]


@pytest.mark.timeout(900)
@pytest.mark.parametrize("ratio,R,steps,full", SWEEP,
                         ids=[f"ratio{r}-R{R}" for r, R, _, _ in SWEEP])
def test_13b_sweep(ratio, R, steps, full):
    from workloads import get_workload
    wl = get_workload("llama2-13b-full")
    keep = [mt for mt in wl.matrices
            if mt.name in ("embed_tokens", "lm_head") or mt.name.startswith("layers.0.")]
    assert sorted({(mt.n, mt.m) for mt in keep}) == [(5120, 5120), (5120, 13824),
                                                     (13824, 5120), (32000, 5120)]
    wl = wl.with_(matrices=tuple(keep), ratio=ratio, refresh=R, accum=4)
    # R = 16 runs with deferred packing (four slots for the S = 4 intervals);
    # R = 1 hands over every step from the score pass, the same launches in
    # both packing modes
    deferred = R > 1
    run_and_check(wl, 4 if deferred else 3, steps, [full], f"13b ratio {ratio} R {R}",
                  deferred=deferred)
