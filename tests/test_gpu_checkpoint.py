"""Checkpoint / resume of the runner: a run interrupted after a mid-interval
step, saved with state_dict, restored into a new runner (new buffers, the
weights restored by the caller) and continued equals the uninterrupted run
bit for bit -- selections, compact states, the packed sums, the offloaded
store and the weights -- in both layouts, with and without the offloaded
optimizer, and with Zen-auto; also a checkpoint taken right after an
interval's first step, resumed with and without the bf16 first-step stage."""
import sys

import numpy as np
import pytest
import torch

from tests._gpu import bits_np
from tests.test_gpu_offload import HP, LAYOUTS, SET, _inputs

pytestmark = pytest.mark.gpu

zf = pytest.importorskip("paper_2505_12242_amd")


def _snapshot(runner):
    out = []
    for q in range(len(runner.shapes)):
        out.append(runner.selection[q].sel_idx.cpu().numpy())
        out.extend(x.cpu().numpy() for x in runner.state[q])
        out.append(runner.acc[q].cpu().numpy())
        if runner.offload:
            out.extend(x.numpy().copy() for x in runner.store[q])
        out.append(bits_np(runner.weights[q]))
    return out


@pytest.mark.timeout(600)
@pytest.mark.parametrize("cut", [7, 5])
@pytest.mark.parametrize("mode", ["plain", "offload", "zen", "zen-offload"])
@pytest.mark.parametrize("layout", LAYOUTS)
def test_resume_equals_uninterrupted_run(layout, mode, cut):
    """cut 5 ends on an interval's first step (R = 4, S = 3: intervals 1-3,
    4, 5-7, ...): with the bf16 first-step stage the checkpoint is taken
    while the interval's values sit in the stage."""
    T_, R, S = 13, 4, 3
    dev = torch.device("cuda")
    slots, _, w, _ = _inputs(SET, T_, 31, layout, dev)
    kw = dict(device=dev, layout=layout, offload="offload" in mode, host_threads=4)
    if "zen" in mode:
        kw["zen_tau"] = 0.8

    def make(weights):
        return zf.SelectiveUpdateRunner(SET, 0.1, HP, R, S, slots, weights, **kw)

    print(f"# checkpoint layout={layout} mode={mode} cut={cut}: uninterrupted", file=sys.stderr, flush=True)
    full = make([x.clone() for x in w])
    for _ in range(T_):
        full.step()
    full.sync()
    want = _snapshot(full)
    full.close()

    print(f"# checkpoint layout={layout} mode={mode} cut={cut}: interrupted", file=sys.stderr, flush=True)
    first_w = [x.clone() for x in w]
    first = make(first_w)
    for _ in range(cut):
        first.step()
    sd = first.state_dict()
    saved_w = [x.clone() for x in first_w]
    first.close()
    del first
    second = make(saved_w)
    second.load_state_dict(sd)
    for _ in range(T_ - cut):
        second.step()
    second.sync()
    got = _snapshot(second)
    second.close()
    assert len(got) == len(want)
    for i, (g, x) in enumerate(zip(got, want)):
        assert g.shape == x.shape and np.array_equal(np.ascontiguousarray(g).view(np.uint8),
                                                     np.ascontiguousarray(x).view(np.uint8)), i


def test_load_rejects_another_configuration():
    dev = torch.device("cuda")
    slots, _, w, _ = _inputs(SET, 2, 31, zf.CHANNEL_MAJOR, dev)
    a = zf.SelectiveUpdateRunner(SET, 0.1, HP, 4, 2, slots, [x.clone() for x in w], device=dev,
                                 layout=zf.CHANNEL_MAJOR)
    a.step()
    sd = a.state_dict()
    b = zf.SelectiveUpdateRunner(SET, 0.1, HP, 4, 4, slots, [x.clone() for x in w], device=dev,
                                 layout=zf.CHANNEL_MAJOR)
    with pytest.raises(ValueError):
        b.load_state_dict(sd)
    a.close()
    b.close()


@pytest.mark.parametrize("save_stage,load_stage", [(False, True), (True, False)])
@pytest.mark.parametrize("layout", LAYOUTS)
def test_resume_across_the_stage_setting(layout, save_stage, load_stage):
    """A checkpoint taken right after an interval's first step by a runner
    with (without) the bf16 first-step stage resumes in a runner without
    (with) it: every later step -- the hand-over at interval ends, else the
    packed sums, the states and W -- equals the uninterrupted run's."""
    T_, cut, R, S = 10, 5, 4, 3
    dev = torch.device("cuda")
    slots, _, w, _ = _inputs(SET, T_, 33, layout, dev)

    def make(weights, stage):
        r = zf.SelectiveUpdateRunner(SET, 0.1, HP, R, S, slots, weights, device=dev,
                                     layout=layout, first_step_stage=stage)
        assert r.use_stage == stage
        return r

    print(f"# checkpoint across stage layout={layout} save={save_stage} load={load_stage}",
          file=sys.stderr, flush=True)
    full = make([x.clone() for x in w], load_stage)
    first_w = [x.clone() for x in w]
    first = make(first_w, save_stage)
    for _ in range(cut):
        full.step()
        first.step()
    sd = first.state_dict()
    saved_w = [x.clone() for x in first_w]
    first.close()
    second = make(saved_w, load_stage)
    second.load_state_dict(sd)
    for t in range(cut + 1, T_ + 1):
        kind = full.step()
        assert second.step() == kind
        torch.cuda.synchronize()
        for q in range(len(SET)):
            pairs = [(bits_np(full.weights[q]), bits_np(second.weights[q]))]
            pairs += [(x.cpu().numpy(), y.cpu().numpy())
                      for x, y in zip(full.state[q], second.state[q])]
            pairs.append((full.unpacked[q].cpu().numpy(), second.unpacked[q].cpu().numpy())
                         if kind.interval_end else
                         (full.acc[q].cpu().numpy(), second.acc[q].cpu().numpy()))
            for i, (a, b) in enumerate(pairs):
                assert np.array_equal(np.ascontiguousarray(a).view(np.uint8),
                                      np.ascontiguousarray(b).view(np.uint8)), (t, q, i)
    full.close()
    second.close()
