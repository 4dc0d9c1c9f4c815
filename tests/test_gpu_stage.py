"""The bf16 first-step stage of the packed buffer (descriptor field
acc_first: channel-major, one bf16 row per channel), through the C ABI, on
the vector and element paths:

* an interval's first step writes the unselected channels' gradient rows to
  their rows of the stage and leaves the fp32 buffer and the selected
  channels' rows untouched; the second step reads the stage and writes
  f32(G1) + f32(G2) to the fp32 buffer, equal bit for bit to the oracle's
  pack_accumulate; the fused hand-over on the second step equals the
  oracle's unpack;
* zf_plan_colnorm_stage: the scores of zf_plan_colnorm plus every channel's
  gradient row in the stage; an Adam-only refresh after it, then the second
  step, equal the plain refresh's results bit for bit;
* zf_plan_colnorm_handover then zf_plan_update_adam_handover (a refresh
  step that is a one-step interval) equal zf_plan_colnorm then
  zf_plan_update_handover bit for bit, from an initial and a remapped state;
* the runner with the stage (its refresh steps through the score pass)
  equals the runner without it bit for bit over six R/S schedules;
* Zen-auto and the separate hand-over pass with the stage equal the same
  runs without it (one-step intervals hand over from the stage,
  zf_plan_unpack_first);
* the row-major stage (one bf16 row per gradient row): first and second
  steps on the 16-byte and per-column kernels, the staged refresh and the
  runner, bit for bit against the runs without it;
* rejected: a stage overlapping the packed buffer, a row-major stage
  without 16-byte rows, Zen-auto on a row-major staged plan, colnorm_stage
  and unpack_first without a stage.
"""
import sys

import numpy as np
import pytest
import torch

import oracle as O
from tests._gpu import bf16_dev, bits_np, f32_np, same_bits
from tests.test_gpu_offload import HP, _inputs, grad_bits, sel_dev
from workloads import derive_seed

pytestmark = pytest.mark.gpu

zf = pytest.importorskip("paper_2505_12242_amd")
CM = zf.CHANNEL_MAJOR


def _buf(rows, cols, dtype, aligned, fill):
    """[rows][cols] storage: 16-byte rows (the vector paths) or an odd
    offset with unpadded rows (the element paths)."""
    if aligned:
        per = 16 // torch.empty(0, dtype=dtype).element_size()
        t = torch.empty(rows, max(per, -(-cols // per) * per), dtype=dtype, device="cuda")
        t = t[:, :cols]
    else:
        t = torch.empty(rows * cols + 1, dtype=dtype, device="cuda")[1:].view(rows, cols)
    t.fill_(fill)
    return t


def _setup(n, m, aligned, ratio=0.1):
    rng = np.random.default_rng(derive_seed("stage", n, m))
    k = O.k_from_ratio(ratio, m)
    sel = O.select_topk(rng.random(m).astype(np.float32), k)
    g = [grad_bits(n, m, derive_seed("stage-g", n, m, t)) for t in (1, 2)]
    G = [bf16_dev(np.ascontiguousarray(x.T)) for x in g]
    return k, sel, g, G


@pytest.mark.parametrize("aligned", [True, False])
@pytest.mark.parametrize("n,m", [(64, 300), (4104, 70), (5, 33), (48, 1000)])
def test_stage_first_and_second_step(n, m, aligned):
    print(f"# stage n={n} m={m} aligned={aligned}", file=sys.stderr, flush=True)
    k, sel, (g1, g2), G = _setup(n, m, aligned)
    u = m - k
    A = _buf(u, n, torch.float32, aligned, np.nan)
    stage = _buf(m, n, torch.bfloat16, aligned, 0.0)
    D = _buf(m, n, torch.float32, True, np.nan)

    def plan(grad, **kw):
        return zf.Plan([zf.MatrixBuffers(grad=grad, k=k, sel=sel_dev(sel), acc=A, unpacked=D,
                                         layout=CM, acc_first=stage, **kw)])

    p1, p2 = plan(G[0]), plan(G[1])
    p1.update(HP, 1, zf.STATES_INPLACE, 1, 4, adam=False, pack=True)
    torch.cuda.synchronize()
    assert torch.isnan(A).all()  # the fp32 buffer is not written on the first step
    st = bits_np(stage)
    uns, sls = sel.unsel.astype(np.int64), sel.sel.astype(np.int64)
    assert np.array_equal(st[uns], np.ascontiguousarray(g1.T)[uns])
    assert (st[sls] == 0).all()  # selected channels' rows untouched
    p2.update(HP, 2, zf.STATES_INPLACE, 2, 4, adam=False, pack=True)
    torch.cuda.synchronize()
    A2 = O.pack_accumulate(g2, sel.unsel, O.pack_accumulate(g1, sel.unsel, None, 1), 2)
    assert same_bits(np.ascontiguousarray(f32_np(A).T), A2)
    # a two-step interval that ends with the fused hand-over: the stage is read
    A.fill_(np.nan)
    p1.update(HP, 1, zf.STATES_INPLACE, 1, 2, adam=False, pack=True)
    Pn, Mn, Vn = (_buf(k, n, torch.float32, True, 0.0) for _ in range(3))
    W = bf16_dev(np.zeros((m, n), np.uint16))
    ph = plan(G[1], weight=W, master=Pn, exp_avg=Mn, exp_avg_sq=Vn)
    ph.update_handover(HP, 2, zf.STATES_INPLACE, 2, 2, 0.5)
    torch.cuda.synchronize()
    assert torch.isnan(A).all()  # the hand-over reads the stage, writes neither buffer
    assert same_bits(np.ascontiguousarray(f32_np(D).T), O.unpack(A2, sel, 0.5))
    for x in (p1, p2, ph):
        x.close()


@pytest.mark.parametrize("aligned", [True, False])
@pytest.mark.parametrize("n,m", [(64, 300), (4104, 70), (5, 33)])
def test_colnorm_stage_then_adam_only_refresh(n, m, aligned):
    """The staged refresh (scores + stage in one pass, Adam-only update) and
    the next step, against the plain refresh (scores, fused update with the
    packing) and the next step: scores, compact states, W and the second
    step's sums bit for bit; the stage holds every channel's gradient row."""
    print(f"# colnorm stage n={n} m={m} aligned={aligned}", file=sys.stderr, flush=True)
    k, sel, (g1, g2), G = _setup(n, m, aligned)
    rng = np.random.default_rng(7)
    W0 = O.bf16_round((rng.standard_normal((n, m)) * 0.02).astype(np.float32))
    outs = []
    for staged in (True, False):
        A = _buf(m - k, n, torch.float32, aligned, np.nan)
        stage = _buf(m, n, torch.bfloat16, aligned, 0.0) if staged else None
        norms = torch.full((m,), np.nan, device="cuda")
        Pn, Mn, Vn = (_buf(k, n, torch.float32, aligned, np.nan) for _ in range(3))
        W = bf16_dev(np.ascontiguousarray(W0.T))
        s = zf.Selection(m, k)
        plans = [zf.Plan([zf.MatrixBuffers(grad=g, k=k, sel=s, weight=W, master=Pn, exp_avg=Mn,
                                           exp_avg_sq=Vn, acc=A, norms=norms, layout=CM,
                                           acc_first=stage)]) for g in G]
        if staged:
            plans[0].colnorm_stage()
        else:
            plans[0].colnorm()
        plans[0].topk_select()
        plans[0].update(HP, 1, zf.STATES_INIT, 1, 4, pack=not staged)
        torch.cuda.synchronize()
        if staged:
            assert np.array_equal(bits_np(stage), np.ascontiguousarray(g1.T))
        plans[1].update(HP, 2, zf.STATES_INPLACE, 2, 4)
        torch.cuda.synchronize()
        outs.append([f32_np(norms), s.sel_idx.cpu().numpy(), f32_np(Pn), f32_np(Mn), f32_np(Vn),
                     bits_np(W), f32_np(A)])
        for p in plans:
            p.close()
    for a, b in zip(*outs):
        assert np.array_equal(np.ascontiguousarray(a).view(np.uint8),
                              np.ascontiguousarray(b).view(np.uint8))


@pytest.mark.parametrize("scale", [1.0, 0.25, 1.0 / 3.0])
@pytest.mark.parametrize("aligned", [True, False])
@pytest.mark.parametrize("n,m", [(64, 300), (2056, 40), (6144, 24), (4101, 20), (5, 33)])
def test_score_pass_handover(n, m, aligned, scale):
    """zf_plan_colnorm_handover alone: every element of the hand-over is
    fp32(scale x widen(g)), one IEEE product (checked with numpy), whatever
    the buffer held before; the scores are those of the plain score pass,
    bit for bit.  The vector path's lanes hand their values to the lanes that
    store them (whole lines per store): shapes with one and several passes,
    a ragged last pass and every lane pair; n % 8 != 0 and unaligned rows
    take the element path."""
    print(f"# score-pass hand-over n={n} m={m} aligned={aligned} scale={scale}",
          file=sys.stderr, flush=True)
    k, sel, (g1, _), G = _setup(n, m, aligned)
    sc = np.float32(scale)
    want = (O.widen(g1) * sc).astype(np.float32)  # [n][m], one product per element
    D = _buf(m, n, torch.float32, aligned, np.nan)
    A = _buf(m - k, n, torch.float32, aligned, np.nan)
    norms = torch.full((m,), np.nan, device="cuda")
    plan = zf.Plan([zf.MatrixBuffers(grad=G[0], k=k, sel=sel_dev(sel), acc=A, norms=norms,
                                     unpacked=D, layout=CM)])
    try:
        plan.colnorm_handover(float(sc))
        torch.cuda.synchronize()
        got_norms = f32_np(norms).copy()
        assert same_bits(f32_np(D).T, want)
        plan.colnorm()
        torch.cuda.synchronize()
        assert same_bits(got_norms, f32_np(norms))
    finally:
        plan.close()


@pytest.mark.parametrize("mode", ["init", "remap"])
@pytest.mark.parametrize("aligned", [True, False])
@pytest.mark.parametrize("n,m", [(64, 300), (4104, 70), (5, 33)])
def test_colnorm_handover_then_adam_handover(n, m, aligned, mode):
    """A refresh step that is a one-step interval, the hand-over taken from
    the score pass (zf_plan_colnorm_handover, selection, then
    zf_plan_update_adam_handover), against the plain path (scores,
    selection, zf_plan_update_handover with step_in_interval 1): scores,
    selection, compact states, W and the hand-over bit for bit."""
    print(f"# colnorm handover n={n} m={m} aligned={aligned} {mode}", file=sys.stderr,
          flush=True)
    k, sel, (g1, g2), G = _setup(n, m, aligned)
    rng = np.random.default_rng(11)
    W0 = O.bf16_round((rng.standard_normal((n, m)) * 0.02).astype(np.float32))
    prev = O.select_topk(rng.random(m).astype(np.float32), k)
    P0 = (rng.standard_normal((k, n)) * 0.02).astype(np.float32)
    outs = []
    for scored in (True, False):
        A = _buf(m - k, n, torch.float32, aligned, np.nan)
        D = _buf(m, n, torch.float32, aligned, np.nan)
        norms = torch.full((m,), np.nan, device="cuda")
        Pn, Mn, Vn = (_buf(k, n, torch.float32, aligned, np.nan) for _ in range(3))
        W = bf16_dev(np.ascontiguousarray(W0.T))
        s = zf.Selection(m, k)
        src = None
        if mode == "remap":
            Pp = torch.from_numpy(P0).cuda()
            src = zf.StateSource(prev=sel_dev(prev), prev_master=Pp, prev_exp_avg=Pp * 0.01,
                                 prev_exp_avg_sq=(Pp * 0.001).abs())
        plan = zf.Plan([zf.MatrixBuffers(grad=G[0], k=k, sel=s, weight=W, master=Pn,
                                         exp_avg=Mn, exp_avg_sq=Vn, acc=A, norms=norms,
                                         unpacked=D, src=src, layout=CM)])
        md = zf.STATES_INIT if mode == "init" else zf.STATES_REMAP
        if scored:
            plan.colnorm_handover(1.0)
            plan.topk_select()
            plan.update_adam_handover(HP, 5, md)
        else:
            plan.colnorm()
            plan.topk_select()
            plan.update_handover(HP, 5, md, 1, 1, 1.0)
        torch.cuda.synchronize()
        outs.append([f32_np(norms), s.sel_idx.cpu().numpy(), f32_np(Pn), f32_np(Mn), f32_np(Vn),
                     bits_np(W), f32_np(D)])
        plan.close()
    for a, b in zip(*outs):
        assert np.array_equal(np.ascontiguousarray(a).view(np.uint8),
                              np.ascontiguousarray(b).view(np.uint8))


@pytest.mark.timeout(600)
@pytest.mark.parametrize("R,S", [(4, 4), (6, 3), (3, 2), (2, 1), (8, 4), (1, 1)])
def test_runner_with_stage_equals_runner_without(R, S):
    T_ = 10
    dev = torch.device("cuda")
    shapes = [(264, 300), (4104, 70), (43, 77), (16, 3), (40, 1500)]
    slots, _, w, _ = _inputs(shapes, T_, 37, CM, dev)
    runs = []
    for stage in (True, False):
        weights = [x.clone() for x in w]
        runner = zf.SelectiveUpdateRunner(shapes, 0.1, HP, R, S, slots, weights, device=dev,
                                          layout=CM, first_step_stage=stage)
        assert runner.use_stage == stage
        out = []
        for t in range(1, T_ + 1):
            print(f"# stage runner R={R} S={S} stage={stage} step {t}", file=sys.stderr,
                  flush=True)
            kind = runner.step()
            torch.cuda.synchronize()
            for q in range(len(shapes)):
                out.append(bits_np(runner.weights[q]))
                out.extend(f32_np(x) for x in runner.state[q])
                if not kind.interval_end:
                    out.append(f32_np(runner.acc[q]))
                else:
                    out.append(f32_np(runner.unpacked[q]))
        runs.append(out)
        runner.close()
    assert len(runs[0]) == len(runs[1])
    for i, (a, b) in enumerate(zip(*runs)):
        assert a.shape == b.shape and np.array_equal(np.ascontiguousarray(a).view(np.uint8),
                                                     np.ascontiguousarray(b).view(np.uint8)), i


def test_plans_that_cannot_use_the_stage_reject_it():
    n, m, k = 8, 64, 6
    rng = np.random.default_rng(3)
    sel = O.select_topk(rng.random(m).astype(np.float32), k)
    # overlapping the packed buffer
    A = torch.zeros((m, n), device="cuda")
    with pytest.raises(RuntimeError):
        zf.Plan([zf.MatrixBuffers(grad=bf16_dev(np.zeros((m, n), np.uint16)), k=k,
                                  sel=sel_dev(sel), acc=A[: m - k], layout=CM,
                                  acc_first=A.view(torch.bfloat16)[:, :n])])
    # colnorm_stage needs a stage
    q = zf.Plan([zf.MatrixBuffers(grad=bf16_dev(np.zeros((m, n), np.uint16)), k=k,
                                  sel=sel_dev(sel), norms=torch.zeros(m, device="cuda"),
                                  layout=CM)])
    with pytest.raises(RuntimeError):
        q.colnorm_stage()
    q.close()


@pytest.mark.timeout(600)
@pytest.mark.parametrize("tau", [0.05, 0.8, float("inf")])
def test_zen_auto_with_stage_equals_without(tau):
    """Zen-auto (statistics fused into the update, separate hand-over pass)
    with the bf16 stage against the same runs without it: interval ends,
    totals, compact states, W, the packed sums and every hand-over bit for
    bit; a small tau ends intervals after one step (the hand-over then reads
    the stage, zf_plan_unpack_first)."""
    T_, R, S = 12, 4, 4
    dev = torch.device("cuda")
    shapes = [(264, 300), (4104, 70), (43, 77), (40, 1500)]
    slots, _, w, _ = _inputs(shapes, T_, 41, CM, dev)
    runs, ends = [], []
    for stage in (True, False):
        weights = [x.clone() for x in w]
        runner = zf.SelectiveUpdateRunner(shapes, 0.1, HP, R, S, slots, weights, device=dev,
                                          layout=CM, zen_tau=tau, first_step_stage=stage)
        assert runner.use_stage == stage and not runner.score_pack
        out, e = [], []
        for t in range(1, T_ + 1):
            print(f"# zen stage tau={tau} stage={stage} step {t}", file=sys.stderr, flush=True)
            kind = runner.step()
            e.append((kind.step_in_interval, kind.interval_end, runner.last_totals.sum_acc,
                      runner.last_totals.sum_sel))
            for q in range(len(shapes)):
                out.append(bits_np(runner.weights[q]))
                out.extend(f32_np(x) for x in runner.state[q])
                out.append(f32_np(runner.unpacked[q]) if kind.interval_end
                           else f32_np(runner.acc[q]))
        runs.append(out)
        ends.append(e)
        runner.close()
    assert ends[0] == ends[1]
    if tau == 0.05:
        assert any(sii == 1 and end for sii, end, _, _ in ends[0][1:])  # one-step intervals
    for i, (a, b) in enumerate(zip(*runs)):
        assert a.shape == b.shape and np.array_equal(np.ascontiguousarray(a).view(np.uint8),
                                                     np.ascontiguousarray(b).view(np.uint8)), i


@pytest.mark.timeout(600)
@pytest.mark.parametrize("R,S", [(4, 4), (2, 1), (6, 3)])
def test_separate_handover_with_stage_equals_without(R, S):
    """The fixed schedule with the separate hand-over pass: with the stage,
    one-step intervals hand over from it (zf_plan_unpack_first)."""
    T_ = 9
    dev = torch.device("cuda")
    shapes = [(264, 300), (43, 77), (16, 3)]
    slots, _, w, _ = _inputs(shapes, T_, 43, CM, dev)
    runs = []
    for stage in (True, False):
        weights = [x.clone() for x in w]
        runner = zf.SelectiveUpdateRunner(shapes, 0.1, HP, R, S, slots, weights, device=dev,
                                          layout=CM, fuse_handover=False, first_step_stage=stage)
        out = []
        for t in range(1, T_ + 1):
            kind = runner.step()
            torch.cuda.synchronize()
            for q in range(len(shapes)):
                out.append(bits_np(runner.weights[q]))
                out.extend(f32_np(x) for x in runner.state[q])
                out.append(f32_np(runner.unpacked[q]) if kind.interval_end
                           else f32_np(runner.acc[q]))
        runs.append(out)
        runner.close()
    for i, (a, b) in enumerate(zip(*runs)):
        assert a.shape == b.shape and np.array_equal(np.ascontiguousarray(a).view(np.uint8),
                                                     np.ascontiguousarray(b).view(np.uint8)), i


@pytest.mark.parametrize("aligned", [True, False])
def test_unpack_first_reads_the_stage(aligned):
    n, m = 40, 300
    k, sel, (g1, _), G = _setup(n, m, aligned)
    A = _buf(m - k, n, torch.float32, aligned, np.nan)
    stage = _buf(m, n, torch.bfloat16, aligned, 0.0)
    D = _buf(m, n, torch.float32, aligned, np.nan)
    plan = zf.Plan([zf.MatrixBuffers(grad=G[0], k=k, sel=sel_dev(sel), acc=A, unpacked=D,
                                     layout=CM, acc_first=stage)])
    plan.update(HP, 1, zf.STATES_INPLACE, 1, 4, adam=False, pack=True)
    plan.unpack_first(0.25)
    torch.cuda.synchronize()
    want = O.unpack(O.pack_accumulate(g1, sel.unsel, None, 1), sel, 0.25)
    assert same_bits(np.ascontiguousarray(f32_np(D).T), want)
    plan.close()
    # a plan without a stage has nothing to read
    p2 = zf.Plan([zf.MatrixBuffers(grad=G[0], k=k, sel=sel_dev(sel), acc=A, unpacked=D,
                                   layout=CM)])
    with pytest.raises(RuntimeError):
        p2.unpack_first(1.0)
    p2.close()


# ------------------------------------------------------------ row-major stage

RM = zf.ROW_MAJOR


@pytest.mark.parametrize("vec", [True, False])
@pytest.mark.parametrize("n,m", [(64, 300), (4104, 70), (5, 33), (48, 1000), (16, 2049)])
def test_row_major_stage_first_and_second_step(n, m, vec):
    """Row-major: the first step stores the gradient rows in the stage (the
    16-byte kernel: whole rows; the per-column kernel, taken when the fp32
    buffer is not 16-byte aligned: the unselected columns), the second step
    reads it; sums and the second-step hand-over bit for bit."""
    print(f"# rm stage n={n} m={m} vec={vec}", file=sys.stderr, flush=True)
    rng = np.random.default_rng(derive_seed("rm-stage", n, m))
    k = O.k_from_ratio(0.1, m)
    sel = O.select_topk(rng.random(m).astype(np.float32), k)
    g1 = grad_bits(n, m, derive_seed("rm-stage-g", n, m, 1))
    g2 = grad_bits(n, m, derive_seed("rm-stage-g", n, m, 2))
    G = [bf16_dev(g, ld=-(-m // 8) * 8) for g in (g1, g2)]
    A = _buf(n, m - k, torch.float32, vec, np.nan)
    stage = _buf(n, m, torch.bfloat16, True, 0.0)
    D = _buf(n, m, torch.float32, vec, np.nan)

    def plan(grad, **kw):
        return zf.Plan([zf.MatrixBuffers(grad=grad, k=k, sel=sel_dev(sel), acc=A, unpacked=D,
                                         layout=RM, acc_first=stage, **kw)])

    p1, p2 = plan(G[0]), plan(G[1])
    p1.update(HP, 1, zf.STATES_INPLACE, 1, 4, adam=False, pack=True)
    torch.cuda.synchronize()
    assert torch.isnan(A).all()
    st = bits_np(stage)
    uns = sel.unsel.astype(np.int64)
    assert np.array_equal(st[:, uns], g1[:, uns])
    p2.update(HP, 2, zf.STATES_INPLACE, 2, 4, adam=False, pack=True)
    torch.cuda.synchronize()
    A2 = O.pack_accumulate(g2, sel.unsel, O.pack_accumulate(g1, sel.unsel, None, 1), 2)
    assert same_bits(f32_np(A), A2)
    A.fill_(np.nan)
    p1.update(HP, 1, zf.STATES_INPLACE, 1, 2, adam=False, pack=True)
    Pn, Mn, Vn = (_buf(n, k, torch.float32, vec, 0.0) for _ in range(3))
    W = bf16_dev(np.zeros((n, m), np.uint16), ld=-(-m // 8) * 8)
    ph = plan(G[1], weight=W, master=Pn, exp_avg=Mn, exp_avg_sq=Vn)
    ph.update_handover(HP, 2, zf.STATES_INPLACE, 2, 2, 0.5)
    torch.cuda.synchronize()
    assert torch.isnan(A).all()
    assert same_bits(f32_np(D), O.unpack(A2, sel, 0.5))
    for x in (p1, p2, ph):
        x.close()


@pytest.mark.parametrize("n,m", [(64, 300), (4104, 70), (5, 33)])
def test_row_major_colnorm_stage_then_adam_only_refresh(n, m):
    print(f"# rm colnorm stage n={n} m={m}", file=sys.stderr, flush=True)
    rng = np.random.default_rng(derive_seed("rm-cs", n, m))
    k = O.k_from_ratio(0.1, m)
    g = [grad_bits(n, m, derive_seed("rm-cs-g", n, m, t)) for t in (1, 2)]
    W0 = O.bf16_round((rng.standard_normal((n, m)) * 0.02).astype(np.float32))
    outs = []
    for staged in (True, False):
        G = [bf16_dev(x, ld=-(-m // 8) * 8) for x in g]
        A = _buf(n, m - k, torch.float32, True, np.nan)
        stage = _buf(n, m, torch.bfloat16, True, 0.0) if staged else None
        norms = torch.full((m,), np.nan, device="cuda")
        Pn, Mn, Vn = (_buf(n, k, torch.float32, True, np.nan) for _ in range(3))
        W = bf16_dev(W0, ld=-(-m // 8) * 8)
        s = zf.Selection(m, k)
        plans = [zf.Plan([zf.MatrixBuffers(grad=x, k=k, sel=s, weight=W, master=Pn, exp_avg=Mn,
                                           exp_avg_sq=Vn, acc=A, norms=norms, layout=RM,
                                           acc_first=stage)]) for x in G]
        if staged:
            plans[0].colnorm_stage()
        else:
            plans[0].colnorm()
        plans[0].topk_select()
        plans[0].update(HP, 1, zf.STATES_INIT, 1, 4, pack=not staged)
        torch.cuda.synchronize()
        if staged:
            assert np.array_equal(bits_np(stage), g[0])
        plans[1].update(HP, 2, zf.STATES_INPLACE, 2, 4)
        torch.cuda.synchronize()
        outs.append([f32_np(norms), s.sel_idx.cpu().numpy(), f32_np(Pn), f32_np(Mn), f32_np(Vn),
                     bits_np(W), f32_np(A)])
        for p in plans:
            p.close()
    for a, b in zip(*outs):
        assert np.array_equal(np.ascontiguousarray(a).view(np.uint8),
                              np.ascontiguousarray(b).view(np.uint8))


@pytest.mark.timeout(600)
@pytest.mark.parametrize("vec", [True, False])
@pytest.mark.parametrize("R,S", [(4, 4), (6, 3), (3, 2), (2, 1)])
def test_row_major_runner_with_stage_equals_runner_without(R, S, vec):
    """vec: every gradient row 16-byte aligned (the plans take the 16-byte
    kernel); else the per-column kernel throughout."""
    T_ = 10
    dev = torch.device("cuda")
    shapes = ([(264, 304), (4104, 72), (40, 1504), (16, 8)] if vec else
              [(264, 300), (4104, 70), (43, 77), (16, 3), (40, 1500)])
    slots, _, w, _ = _inputs(shapes, T_, 47, RM, dev)
    runs = []
    for stage in (True, False):
        weights = [x.clone() for x in w]
        runner = zf.SelectiveUpdateRunner(shapes, 0.1, HP, R, S, slots, weights, device=dev,
                                          layout=RM, first_step_stage=stage)
        assert runner.use_stage == stage and not runner.score_handover
        out = []
        for t in range(1, T_ + 1):
            print(f"# rm stage runner R={R} S={S} vec={vec} stage={stage} step {t}", file=sys.stderr,
                  flush=True)
            kind = runner.step()
            torch.cuda.synchronize()
            for q in range(len(shapes)):
                out.append(bits_np(runner.weights[q]))
                out.extend(f32_np(x) for x in runner.state[q])
                out.append(f32_np(runner.unpacked[q]) if kind.interval_end
                           else f32_np(runner.acc[q]))
        runs.append(out)
        runner.close()
    for i, (a, b) in enumerate(zip(*runs)):
        assert a.shape == b.shape and np.array_equal(np.ascontiguousarray(a).view(np.uint8),
                                                     np.ascontiguousarray(b).view(np.uint8)), i


def test_row_major_stage_rules():
    n, m, k = 8, 64, 6
    rng = np.random.default_rng(3)
    sel = O.select_topk(rng.random(m).astype(np.float32), k)
    base = dict(grad=bf16_dev(np.zeros((n, m), np.uint16)), k=k, sel=sel_dev(sel),
                acc=torch.zeros((n, m - k), device="cuda"), layout=RM)
    # the row-major stage must have 16-byte rows
    odd = torch.zeros(n * m + 1, dtype=torch.bfloat16, device="cuda")[1:].view(n, m)
    with pytest.raises(RuntimeError):
        zf.Plan([zf.MatrixBuffers(acc_first=odd, **base)])
    # Zen-auto rejects a row-major plan with a stage
    z = zf.Plan([zf.MatrixBuffers(acc_first=torch.zeros((n, m), dtype=torch.bfloat16,
                                                        device="cuda"),
                                  weight=bf16_dev(np.zeros((n, m), np.uint16)),
                                  master=torch.zeros((n, k), device="cuda"),
                                  exp_avg=torch.zeros((n, k), device="cuda"),
                                  exp_avg_sq=torch.zeros((n, k), device="cuda"),
                                  sel_sq=torch.zeros(k, device="cuda"),
                                  acc_sq=torch.zeros(m - k, device="cuda"), **base)])
    totals = torch.zeros(zf.ZEN_TOTALS_BYTES // 8, dtype=torch.int64, device="cuda")
    with pytest.raises(RuntimeError):
        z.update_zen(HP, 1, zf.STATES_INPLACE, 1, 4, 1.0, totals)
    z.close()


@pytest.mark.parametrize("master", [False, True])
@pytest.mark.parametrize("mode", ["init", "remap"])
def test_row_major_adam_only_selected_grid(mode, master):
    """Row-major Adam alone (the staged refresh's update): states and W equal
    the fused per-column pass's bit for bit, over a batched plan whose
    matrices span one to many column tiles and ragged row blocks (0 selected
    columns included)."""
    shapes = [(300, 2900), (17, 77), (4104, 70), (9, 5000), (6, 40)]
    ratios = [0.1, 0.1, 0.1, 0.2, 0.0]
    print(f"# rm selected grid mode={mode} master={master}", file=sys.stderr, flush=True)
    rng = np.random.default_rng(derive_seed("rm-selg", mode, master))
    res = []
    for pack in (False, True):
        bufs = []
        for (n, m), ratio in zip(shapes, ratios):
            k = O.k_from_ratio(ratio, m)
            r2 = np.random.default_rng(derive_seed("rm-selg-q", n, m))
            old = O.select_topk(r2.random(m).astype(np.float32), k)
            new = O.select_topk(r2.random(m).astype(np.float32), k)
            g = grad_bits(n, m, derive_seed("rm-selg-g", n, m))
            W = O.bf16_round((r2.standard_normal((n, m)) * 0.02).astype(np.float32))
            prev = [(r2.standard_normal((n, k)) * s).astype(np.float32) for s in (0.02, 1e-3, 1e-3)]
            prev[2] = np.abs(prev[2])
            ld_m = -(-m // 8) * 8
            dev = lambda x: _buf(n, x.shape[1], torch.float32, True, 0.0).copy_(torch.from_numpy(x))
            P, M, V = (_buf(n, k, torch.float32, True, np.nan) for _ in range(3))
            src = None
            if mode == "remap" or master:
                src = zf.StateSource(
                    prev=sel_dev(old) if mode == "remap" else None,
                    prev_master=dev(prev[0]) if mode == "remap" else None,
                    prev_exp_avg=dev(prev[1]) if mode == "remap" else None,
                    prev_exp_avg_sq=dev(prev[2]) if mode == "remap" else None,
                    init_master=dev(W + np.float32(1e-3)) if master else None)
            bufs.append(zf.MatrixBuffers(
                grad=bf16_dev(g, ld=ld_m), k=k, sel=sel_dev(new), weight=bf16_dev(W, ld=ld_m),
                master=P, exp_avg=M, exp_avg_sq=V, src=src, layout=RM,
                acc=_buf(n, m - k, torch.float32, False, 0.0)))
        plan = zf.Plan(bufs)
        plan.update(HP, 3, zf.STATES_INIT if mode == "init" else zf.STATES_REMAP, 1, 4,
                    pack=pack)
        torch.cuda.synchronize()
        res.append([x for b in bufs for x in (f32_np(b.master), f32_np(b.exp_avg),
                                              f32_np(b.exp_avg_sq), bits_np(b.weight))])
        plan.close()
    for i, (a, b) in enumerate(zip(*res)):
        assert np.array_equal(np.ascontiguousarray(a).view(np.uint8),
                              np.ascontiguousarray(b).view(np.uint8)), i
