"""End-to-end parity of the batched step driver with the oracle on the
single 4096x4096 linear weight (one fresh-selection step) and on one
Llama-2-7B decoder layer (4 steps: selection at step 1 reused, unselected
columns accumulated, hand-over at step 4): every output compared in full."""
import numpy as np
import pytest
import torch

import oracle as O
from tests._gpu import bf16_dev, bits_np, f32_np, mask_np, rel_close, same_bits
from workloads import derive_seed, get_workload, gradient, master_weights, step_scales

pytestmark = pytest.mark.gpu

zf = pytest.importorskip("paper_2505_12242_amd")


def run_workload(name, use_master):
    wl = get_workload(name)
    hp = zf.AdamHparams(wl.hyper.lr, wl.hyper.beta1, wl.hyper.beta2, wl.hyper.eps,
                        wl.hyper.weight_decay)
    shapes = [(mt.n, mt.m) for mt in wl.matrices]
    ks = [O.k_from_ratio(wl.ratio, m) for _, m in shapes]
    dev = torch.device("cuda")
    slots, weights, masters = [], [], []
    for t in range(1, wl.steps + 1):
        slot = []
        for q, (n, m) in enumerate(shapes):
            s = step_scales(wl, q, t, k_boundary=ks[q])
            slot.append(gradient(n, m, s, derive_seed(wl.seed, q, "grad", t), device=dev))
        slots.append(slot)
    for q, (n, m) in enumerate(shapes):
        mw = master_weights(n, m, derive_seed(wl.seed, q, "master"), wl.master_std, device=dev)
        masters.append(mw)
        weights.append(mw.to(torch.bfloat16))
    w0 = [bits_np(w) for w in weights]
    runner = zf.SelectiveUpdateRunner(shapes, wl.ratio, hp, wl.refresh, wl.accum, slots, weights,
                                      init_master=masters if use_master else None)
    orcs = [O.MatrixOracle(f32_np(masters[q]) if use_master else O.widen(w0[q]), w0[q], wl.ratio,
                           hp.lr, hp.beta1, hp.beta2, hp.eps, hp.weight_decay, wl.refresh,
                           wl.accum) for q in range(len(shapes))]
    for t in range(1, wl.steps + 1):
        kind = runner.step()
        torch.cuda.synchronize()
        for q, orc in enumerate(orcs):
            out = orc.step(bits_np(slots[t - 1][q]))
            name_q = wl.matrices[q].name
            if kind.refresh:
                ok, worst = rel_close(f32_np(runner.norms[q]), out["norms"], 1e-5)
                assert ok, (name_q, t, worst)
                sel = runner.selection[q]
                assert np.array_equal(sel.sel_idx.cpu().numpy(), orc.sel.sel), (name_q, t)
                assert np.array_equal(sel.unsel_idx.cpu().numpy(), orc.sel.unsel), (name_q, t)
                assert np.array_equal(mask_np(sel.mask), orc.sel.mask), (name_q, t)
                assert np.array_equal(sel.prefix.cpu().numpy(), orc.sel.prefix), (name_q, t)
            assert same_bits(f32_np(runner.acc[q]), orc.A), (name_q, t)
            P, M, V = (f32_np(x) for x in runner.state[q])
            ok, w = rel_close(P, orc.P, 2e-6)
            assert ok, (name_q, t, "P", w)
            ok, w = rel_close(V, orc.V, 2e-6)
            assert ok, (name_q, t, "V", w)
            assert same_bits(P, orc.P) and same_bits(M, orc.M) and same_bits(V, orc.V), (name_q, t)
            assert np.array_equal(bits_np(weights[q]), orc.W), (name_q, t)
            if kind.interval_end:
                assert same_bits(f32_np(runner.unpacked[q]), out["unpacked"]), (name_q, t)
    runner.close()


@pytest.mark.timeout(300)
def test_linear_4096_fresh_selection_step():
    run_workload("linear-4096x4096", use_master=True)


@pytest.mark.timeout(900)
def test_llama2_7b_layer_four_steps():
    run_workload("llama2-7b-layer", use_master=False)
