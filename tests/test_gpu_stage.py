"""The bf16 first-step stage of the packed buffer (channel-major plans,
descriptor field acc_first), through the C ABI:

* an interval's first step writes the unselected channels' gradient bits to
  the stage and leaves the fp32 buffer untouched; the second step reads the
  stage and writes f32(G1) + f32(G2) to the fp32 buffer, equal bit for bit to
  the oracle's pack_accumulate; the fused hand-over on the second step equals
  the oracle's unpack;
* the runner with the stage equals the runner without it bit for bit (W,
  compact states, packed sums, hand-over) over intervals of 1 to 4 steps,
  with vector and element paths;
* plans that cannot use it reject it: row-major descriptors at creation,
  unpack / Zen-auto / pending refresh on a plan that has one.
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


@pytest.mark.parametrize("n,m", [(64, 300), (4104, 70), (5, 33), (2048, 1000)])
def test_stage_first_and_second_step(n, m):
    print(f"# stage n={n} m={m}", file=sys.stderr, flush=True)
    rng = np.random.default_rng(derive_seed("stage", n, m))
    k = O.k_from_ratio(0.1, m)
    sel = O.select_topk(rng.random(m).astype(np.float32), k)
    u = m - k
    g1 = grad_bits(n, m, derive_seed("stage-g", n, m, 1))
    g2 = grad_bits(n, m, derive_seed("stage-g", n, m, 2))
    A = torch.full((u, n), np.nan, device="cuda")
    stage = torch.zeros((u, n), dtype=torch.bfloat16, device="cuda")
    D = torch.full((m, n), np.nan, device="cuda")
    G = [bf16_dev(np.ascontiguousarray(g.T)) for g in (g1, g2)]

    def plan(grad):
        return zf.Plan([zf.MatrixBuffers(grad=grad, k=k, sel=sel_dev(sel), acc=A, unpacked=D,
                                         layout=CM, acc_first=stage)])

    p1, p2 = plan(G[0]), plan(G[1])
    p1.update(HP, 1, zf.STATES_INPLACE, 1, 4, adam=False, pack=True)
    torch.cuda.synchronize()
    assert torch.isnan(A).all()  # the fp32 buffer is not written on the first step
    want_stage = np.ascontiguousarray(g1[:, sel.unsel.astype(np.int64)].T)
    assert np.array_equal(bits_np(stage), want_stage)
    p2.update(HP, 2, zf.STATES_INPLACE, 2, 4, adam=False, pack=True)
    torch.cuda.synchronize()
    A2 = O.pack_accumulate(g2, sel.unsel, O.pack_accumulate(g1, sel.unsel, None, 1), 2)
    assert same_bits(np.ascontiguousarray(f32_np(A).T), A2)
    # a two-step interval that ends with the fused hand-over: the stage is read
    A.fill_(np.nan)
    p1.update(HP, 1, zf.STATES_INPLACE, 1, 2, adam=False, pack=True)
    Pn = torch.zeros((k, n), device="cuda")
    Mn, Vn = torch.zeros_like(Pn), torch.zeros_like(Pn)
    W = bf16_dev(np.zeros((m, n), np.uint16))
    ph = zf.Plan([zf.MatrixBuffers(grad=G[1], k=k, sel=sel_dev(sel), acc=A, unpacked=D,
                                   weight=W, master=Pn, exp_avg=Mn, exp_avg_sq=Vn, layout=CM,
                                   acc_first=stage)])
    ph.update_handover(HP, 2, zf.STATES_INPLACE, 2, 2, 0.5)
    torch.cuda.synchronize()
    assert torch.isnan(A).all()  # the hand-over reads the stage, writes neither buffer
    assert same_bits(np.ascontiguousarray(f32_np(D).T), O.unpack(A2, sel, 0.5))
    for x in (p1, p2, ph):
        x.close()


@pytest.mark.timeout(600)
@pytest.mark.parametrize("R,S", [(4, 4), (6, 3), (3, 2), (2, 1), (8, 4)])
def test_runner_with_stage_equals_runner_without(R, S):
    T_ = 10
    dev = torch.device("cuda")
    slots, _, w, _ = _inputs([(264, 300), (4104, 70), (43, 77), (16, 3)], T_, 37, CM, dev)
    shapes = [(264, 300), (4104, 70), (43, 77), (16, 3)]
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
        assert a.shape == b.shape and np.array_equal(a.view(np.uint8), b.view(np.uint8)), i


def test_plans_that_cannot_use_the_stage_reject_it():
    n, m, k = 8, 64, 6
    rng = np.random.default_rng(3)
    sel = O.select_topk(rng.random(m).astype(np.float32), k)
    stage_cm = torch.zeros((m - k, n), dtype=torch.bfloat16, device="cuda")
    # row-major descriptors may not give one
    with pytest.raises(RuntimeError):
        zf.Plan([zf.MatrixBuffers(grad=bf16_dev(np.zeros((n, m), np.uint16)), k=k,
                                  sel=sel_dev(sel), acc=torch.zeros((n, m - k), device="cuda"),
                                  layout=zf.ROW_MAJOR,
                                  acc_first=torch.zeros((n, m - k), dtype=torch.bfloat16,
                                                        device="cuda"))])
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
