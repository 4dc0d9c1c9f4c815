"""Adam at its numerical edges on the device, bit for bit against the oracle
(the selective optimizer extends PyTorch's fp32 Adam: Implementation,
"Selective GPU-side Optimizer"; Adam of Kingma & Ba).

Gradients are bf16 patterns over the whole exponent range, by class: +-0
(the denominator is eps exactly), |g| around 1e-9 .. 1e-7 (eps decides the
denominator), |g| < 2^-64 including bf16 subnormals (C2 * g^2 subnormal or
zero), |g| >= 2^64 (g * g overflows), any finite pattern.  States take zero,
subnormal, eps-sized, typical and huge values (second moments >= 0, -0.0
included; masters at bf16 rounding ties and near-ties), and in a second
variant infinities in some moments, so that some steps divide infinity by
infinity.  Each element of the result is compared bit for bit; where the
oracle gives NaN the device must give NaN (payloads are not compared).

Every device path runs: zf_adam_selected, zf_update_fused (an interval's
first step and an accumulating step) and zf_update_fused_handover, plus
zf_adam_selected from an fp32 master (ZF_STATES_INIT), each in both
layouts, on 16-byte aligned storage (the channel-major vector path, the
row-major 16-byte kernel) and on storage offset by one element (the
channel-major element path, the row-major per-column kernel); with and
without decoupled weight decay; at steps 1 and 1000.  This also stands in
for a check that the device square root and division are correctly rounded
and that no operation is contracted or flushed to zero: any of those would
change bits somewhere in these ranges.
"""
import numpy as np
import pytest
import torch

import oracle as O
from tests._edges import bf16_as_f32, first_mismatch, inputs, same_nan_aware
from tests.test_gpu_random_cases import Bufs

pytestmark = pytest.mark.gpu

zf = pytest.importorskip("paper_2505_12242_amd")

# n a multiple of 8 (channel-major vector path when aligned); m = 1100 spans
# two tiles of the row-major 16-byte kernel
SHAPES = [(72, 300, 0.3), (16, 1100, 0.1)]
ENTRIES = ["adam", "fused-first", "fused-accumulate", "handover", "init"]


def to_dev_selection(s: O.Selection):
    out = zf.Selection(s.m, s.k)
    out.sel_idx.copy_(torch.from_numpy(s.sel.astype(np.int32)))
    out.unsel_idx.copy_(torch.from_numpy(s.unsel.astype(np.int32)))
    out.mask.copy_(torch.from_numpy(s.mask.view(np.int64)))
    out.prefix.copy_(torch.from_numpy(s.prefix.astype(np.int32)))
    return out


@pytest.mark.parametrize("nonfinite", [False, True], ids=["finite", "inf-moments"])
@pytest.mark.parametrize("step", [1, 1000])
@pytest.mark.parametrize("wd", [0.0, 0.01])
@pytest.mark.parametrize("entry", ENTRIES)
@pytest.mark.parametrize("aligned", [True, False], ids=["vec", "elem"])
@pytest.mark.parametrize("layout", [zf.ROW_MAJOR, zf.CHANNEL_MAJOR], ids=["rm", "cm"])
@pytest.mark.parametrize("n,m,ratio", SHAPES)
def test_adam_edges(n, m, ratio, layout, aligned, entry, wd, step, nonfinite):
    G, sel, P, Mo, V, W, A, master = inputs(n, m, ratio, step + 7 * int(nonfinite), nonfinite)
    hp = zf.AdamHparams(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=wd)
    c = O.AdamConsts.at_step(hp.lr, hp.beta1, hp.beta2, hp.eps, hp.weight_decay, step)
    B = Bufs(layout, aligned)
    Gd, Wd = B.bf16(G), B.bf16(W)
    sd = to_dev_selection(sel)
    k = sel.k
    if entry == "init":
        Pd, Md, Vd = (B.f32(np.full((n, k), np.nan, np.float32)) for _ in range(3))
    else:
        Pd, Md, Vd = B.f32(P), B.f32(Mo), B.f32(V)
    Ad = B.f32(A)
    sii = 1 if entry == "fused-first" else 2
    scale = float(np.float32(1.0 / 3.0))
    D = None
    if entry == "adam":
        zf.adam_selected(Gd, sd, Pd, Md, Vd, Wd, hp, step, layout=layout)
    elif entry == "init":
        src = zf.StateSource(init_master=B.f32(master))
        zf.adam_selected(Gd, sd, Pd, Md, Vd, Wd, hp, step, mode=zf.STATES_INIT, src=src,
                         layout=layout)
    elif entry.startswith("fused"):
        zf.update_fused(Gd, sd, Pd, Md, Vd, Wd, hp, step, Ad, sii, 4, layout=layout)
    else:
        D = B.f32(np.full((n, m), np.nan, np.float32))
        zf.update_fused_handover(Gd, sd, Pd, Md, Vd, Wd, hp, step, Ad, sii, 4, scale, out=D,
                                 layout=layout)
    torch.cuda.synchronize()

    with np.errstate(all="ignore"):
        if entry == "init":
            P0, M0, V0 = O.remap(None, sel, None, None, None, W, master)
        else:
            P0, M0, V0 = P, Mo, V
        Pw, Mw, Vw, wsel = O.adam_selected(G, sel.sel, P0, M0, V0, c)
        Ww = W.copy()
        Ww[:, sel.sel.astype(np.int64)] = wsel
        if entry.startswith("fused"):
            Aw = O.pack_accumulate(G, sel.unsel, A, sii)
        if entry == "handover":
            Dw = O.unpack(O.pack_accumulate(G, sel.unsel, A, sii), sel, scale)

    case = (n, m, "rm" if layout == zf.ROW_MAJOR else "cm", aligned, entry, wd, step)
    for name, dev, want in (("P", Pd, Pw), ("M", Md, Mw), ("V", Vd, Vw)):
        got = B.logical(dev)
        assert same_nan_aware(got, want), (case, name, first_mismatch(got, want))
    Wg = B.logical(Wd)
    assert same_nan_aware(bf16_as_f32(Wg), bf16_as_f32(Ww)), \
        (case, "W", first_mismatch(bf16_as_f32(Wg), bf16_as_f32(Ww)))
    if entry.startswith("fused"):
        assert same_nan_aware(B.logical(Ad), Aw), (case, "A", first_mismatch(B.logical(Ad), Aw))
    else:
        assert np.array_equal(B.logical(Ad).view(np.uint32), A.view(np.uint32)), (case, "A")
    if D is not None:
        assert same_nan_aware(B.logical(D), Dw), (case, "D", first_mismatch(B.logical(D), Dw))
