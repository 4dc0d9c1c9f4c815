"""The bf16 first-step stage of the packed buffer (descriptor field
acc_first), through the C ABI, in both layouts and on the vector and
element paths:

* an interval's first step writes the unselected channels' gradient bits to
  the stage and leaves the fp32 buffer untouched; the second step reads the
  stage and writes f32(G1) + f32(G2) to the fp32 buffer, equal bit for bit to
  the oracle's pack_accumulate; the fused hand-over on the second step equals
  the oracle's unpack;
* the runner with the stage equals the runner without it bit for bit (W,
  compact states, packed sums, hand-over) over intervals of 1 to 4 steps,
  with vector and element paths;
* a stage overlapping the packed buffer is rejected at plan creation, and
  the separate hand-over pass on a plan that has one.
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


def _buf(layout, rows_l, cols_l, dtype, aligned, fill):
    """Storage of a logical rows_l x cols_l matrix: 16-byte rows (the vector
    paths) or an odd offset with unpadded rows (the element paths)."""
    shape = (rows_l, cols_l) if layout == zf.ROW_MAJOR else (cols_l, rows_l)
    if aligned:
        t = zf.alloc_stored(layout, rows_l, cols_l, dtype, "cuda")
    else:
        t = torch.empty(shape[0] * shape[1] + 1, dtype=dtype, device="cuda")[1:].view(*shape)
    t.fill_(fill)
    return t


def _logical(t, layout):
    a = t.cpu()
    a = a if layout == zf.ROW_MAJOR else a.t()
    return a.contiguous()


@pytest.mark.parametrize("aligned", [True, False])
@pytest.mark.parametrize("n,m", [(64, 300), (4104, 70), (5, 33), (48, 1000)])
@pytest.mark.parametrize("layout", [zf.ROW_MAJOR, CM], ids=["rm", "cm"])
def test_stage_first_and_second_step(layout, n, m, aligned):
    print(f"# stage layout={layout} n={n} m={m} aligned={aligned}", file=sys.stderr, flush=True)
    rng = np.random.default_rng(derive_seed("stage", n, m))
    k = O.k_from_ratio(0.1, m)
    sel = O.select_topk(rng.random(m).astype(np.float32), k)
    u = m - k
    g1 = grad_bits(n, m, derive_seed("stage-g", n, m, 1))
    g2 = grad_bits(n, m, derive_seed("stage-g", n, m, 2))
    A = _buf(layout, n, u, torch.float32, aligned, np.nan)
    stage = _buf(layout, n, u, torch.bfloat16, aligned, 0.0)
    D = _buf(layout, n, m, torch.float32, True, np.nan)
    T = (lambda a: a) if layout == zf.ROW_MAJOR else (lambda a: np.ascontiguousarray(a.T))
    G = [bf16_dev(T(g)) for g in (g1, g2)]

    def plan(grad, **kw):
        return zf.Plan([zf.MatrixBuffers(grad=grad, k=k, sel=sel_dev(sel), acc=A, unpacked=D,
                                         layout=layout, acc_first=stage, **kw)])

    p1, p2 = plan(G[0]), plan(G[1])
    p1.update(HP, 1, zf.STATES_INPLACE, 1, 4, adam=False, pack=True)
    torch.cuda.synchronize()
    assert torch.isnan(A).all()  # the fp32 buffer is not written on the first step
    want_stage = np.ascontiguousarray(g1[:, sel.unsel.astype(np.int64)])
    assert np.array_equal(bits_np(_logical(stage, layout)), want_stage)
    p2.update(HP, 2, zf.STATES_INPLACE, 2, 4, adam=False, pack=True)
    torch.cuda.synchronize()
    A2 = O.pack_accumulate(g2, sel.unsel, O.pack_accumulate(g1, sel.unsel, None, 1), 2)
    assert same_bits(f32_np(_logical(A, layout)), A2)
    # a two-step interval that ends with the fused hand-over: the stage is read
    A.fill_(np.nan)
    p1.update(HP, 1, zf.STATES_INPLACE, 1, 2, adam=False, pack=True)
    Pn = _buf(layout, n, k, torch.float32, True, 0.0)
    Mn, Vn = _buf(layout, n, k, torch.float32, True, 0.0), _buf(layout, n, k, torch.float32,
                                                                True, 0.0)
    W = bf16_dev(np.zeros((n, m) if layout == zf.ROW_MAJOR else (m, n), np.uint16))
    ph = plan(G[1], weight=W, master=Pn, exp_avg=Mn, exp_avg_sq=Vn)
    ph.update_handover(HP, 2, zf.STATES_INPLACE, 2, 2, 0.5)
    torch.cuda.synchronize()
    assert torch.isnan(A).all()  # the hand-over reads the stage, writes neither buffer
    assert same_bits(f32_np(_logical(D, layout)), O.unpack(A2, sel, 0.5))
    for x in (p1, p2, ph):
        x.close()


@pytest.mark.timeout(600)
@pytest.mark.parametrize("R,S", [(4, 4), (6, 3), (3, 2), (2, 1), (8, 4)])
@pytest.mark.parametrize("layout", [zf.ROW_MAJOR, CM], ids=["rm", "cm"])
def test_runner_with_stage_equals_runner_without(layout, R, S):
    T_ = 10
    dev = torch.device("cuda")
    shapes = [(264, 300), (4104, 70), (43, 77), (16, 3), (40, 1500)]
    slots, _, w, _ = _inputs(shapes, T_, 37, layout, dev)
    runs = []
    for stage in (True, False):  # True: also in the row-major layout
        weights = [x.clone() for x in w]
        runner = zf.SelectiveUpdateRunner(shapes, 0.1, HP, R, S, slots, weights, device=dev,
                                          layout=layout, first_step_stage=stage)
        assert runner.use_stage == stage
        out = []
        for t in range(1, T_ + 1):
            print(f"# stage runner layout={layout} R={R} S={S} stage={stage} step {t}",
                  file=sys.stderr, flush=True)
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
    stage_cm = torch.zeros((m - k, n), dtype=torch.bfloat16, device="cuda")
    # overlapping the packed buffer
    A = torch.zeros((m - k, n), device="cuda")
    with pytest.raises(RuntimeError):
        zf.Plan([zf.MatrixBuffers(grad=bf16_dev(np.zeros((m, n), np.uint16)), k=k,
                                  sel=sel_dev(sel), acc=A, layout=CM,
                                  acc_first=A.view(torch.bfloat16)[:, :n])])
    D = torch.zeros((m, n), device="cuda")
    p = zf.Plan([zf.MatrixBuffers(grad=bf16_dev(np.zeros((m, n), np.uint16)), k=k,
                                  sel=sel_dev(sel), acc=A, unpacked=D, layout=CM,
                                  acc_first=stage_cm)])
    with pytest.raises(RuntimeError):
        p.unpack(1.0)
    p.close()
