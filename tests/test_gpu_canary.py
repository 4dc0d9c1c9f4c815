"""Out-of-bounds write guards: every output of every entry point lives inside
a larger device buffer whose words before and after it, and whose row
padding (ld > width), hold a sentinel bit pattern; after each call every
sentinel must be intact.  Ragged shapes take the element-wise paths as well
as the 16-byte paths, in both layouts.  Outputs are also checked to be fully
written where they must be (no sentinel left inside the written region)."""
import numpy as np
import pytest
import torch

import oracle as O
from workloads import derive_seed, gradient

pytestmark = pytest.mark.gpu

zf = pytest.importorskip("paper_2505_12242_amd")
HP = zf.AdamHparams(lr=1e-3)
LAYOUTS = [pytest.param(zf.ROW_MAJOR, id="rm"), pytest.param(zf.CHANNEL_MAJOR, id="cm")]
SENT32 = 0x7FBADBAD  # a NaN pattern no kernel output here produces
SENT16 = 0x7FBB
GUARD = 64           # sentinel elements before and after each output


class Guarded:
    """A rows x width view (row stride ld = width + pad) inside a buffer with
    GUARD sentinel elements on both sides; dtype float32 or bfloat16."""

    def __init__(self, rows, width, dtype):
        self.rows, self.width, self.dtype = rows, width, dtype
        # padded rows that keep 16-byte alignment (the vector paths stay in use
        # whenever the width allows them)
        self.ld = ((width + 7) // 8) * 8 + 8 if rows > 1 else width
        total = GUARD * 2 + max(rows, 1) * self.ld
        itype = torch.int32 if dtype == torch.float32 else torch.int16
        sent = SENT32 if dtype == torch.float32 else SENT16
        self.raw = torch.full((total,), sent, dtype=itype, device="cuda")
        self.sent = sent
        body = self.raw[GUARD: GUARD + max(rows, 1) * self.ld].view(dtype)
        self.t = body.view(max(rows, 1), self.ld)[:rows, :width]

    def fill(self, array):
        a = np.ascontiguousarray(array)
        if self.dtype == torch.bfloat16:
            t = torch.from_numpy(a.view(np.int16)).view(torch.bfloat16)
        else:
            t = torch.from_numpy(a.astype(np.float32))
        self.t.copy_(t.to("cuda"))
        return self

    def intact(self) -> bool:
        r = self.raw.cpu().numpy()
        if not (np.all(r[:GUARD] == self.sent) and np.all(r[-GUARD:] == self.sent)):
            return False
        if self.rows > 1 and self.ld > self.width:
            body = r[GUARD: GUARD + self.rows * self.ld].reshape(self.rows, self.ld)
            if not np.all(body[:, self.width:] == self.sent):
                return False
        return True

    def fully_written(self) -> bool:
        raw = self.t.contiguous().view(torch.int32 if self.dtype == torch.float32 else torch.int16)
        return not bool((raw.cpu() == self.sent).any())


def storage(layout, rows_l, cols_l):
    return (rows_l, cols_l) if layout == zf.ROW_MAJOR else (cols_l, rows_l)


def grad_bits(n, m, seed):
    g = torch.Generator().manual_seed(seed)
    s = torch.exp(1.5 * torch.randn(m, generator=g, dtype=torch.float64))
    return gradient(n, m, s, seed=seed).view(torch.int16).numpy().view(np.uint16)


def to_layout(a, layout):
    return a if layout == zf.ROW_MAJOR else np.ascontiguousarray(a.T)


@pytest.mark.parametrize("n,m,ratio", [(1, 1, 1.0), (3, 7, 0.3), (43, 77, 0.1), (64, 130, 0.1),
                                       (264, 300, 0.1), (4104, 70, 0.1)])
@pytest.mark.parametrize("layout", LAYOUTS)
def test_no_write_outside_outputs(n, m, ratio, layout):
    bits = grad_bits(n, m, derive_seed("canary", n, m))
    G = Guarded(*storage(layout, n, m), torch.bfloat16).fill(to_layout(bits, layout))
    # scores
    norms = Guarded(1, m, torch.float32)
    zf.colnorm(G.t, out=norms.t.view(m), layout=layout,
               workspace=torch.zeros(max(zf.colnorm_workspace_bytes(n, m, layout), 8),
                                     dtype=torch.uint8, device="cuda"))
    torch.cuda.synchronize()
    assert norms.intact() and norms.fully_written()
    # selection
    k = zf.k_from_ratio(ratio, m)
    sel = zf.Selection(m, k)
    gs = [Guarded(1, k, torch.float32), Guarded(1, m - k, torch.float32)]
    sel.sel_idx = gs[0].t.view(k).view(torch.int32)
    sel.unsel_idx = gs[1].t.view(m - k).view(torch.int32)
    zf.topk_select(norms.t.view(m), ratio, out=sel)
    torch.cuda.synchronize()
    assert all(g.intact() for g in gs)
    # Adam (init), pack, fused pass, hand-over, scatter
    rng = np.random.default_rng(n + m)
    W = Guarded(*storage(layout, n, m), torch.bfloat16).fill(
        to_layout(O.bf16_round((rng.standard_normal((n, m)) * 0.02).astype(np.float32)), layout))
    P, M, V = (Guarded(*storage(layout, n, k), torch.float32) for _ in range(3))
    zf.adam_selected(G.t, sel, P.t, M.t, V.t, W.t, HP, 1, mode=zf.STATES_INIT, layout=layout)
    A = Guarded(*storage(layout, n, m - k), torch.float32)
    zf.pack_accumulate(G.t, sel, A.t, 1, 4, layout=layout)
    torch.cuda.synchronize()
    for g in (P, M, V, W, A):
        assert g.intact()
    for g in (P, M, V, A):
        assert g.fully_written()
    zf.update_fused(G.t, sel, P.t, M.t, V.t, W.t, HP, 2, A.t, 2, 4, layout=layout)
    D = Guarded(*storage(layout, n, m), torch.float32)
    zf.unpack(A.t, sel, 0.5, out=D.t, layout=layout)
    D2 = Guarded(*storage(layout, n, m), torch.float32)
    zf.update_fused_handover(G.t, sel, P.t, M.t, V.t, W.t, HP, 3, A.t, 3, 4, 1.0 / 3.0,
                             out=D2.t, layout=layout)
    torch.cuda.synchronize()
    for g in (P, M, V, W, A, D, D2):
        assert g.intact()
    assert D.fully_written() and D2.fully_written()
    cols = Guarded(*storage(layout, n, m - k), torch.bfloat16).fill(
        to_layout(O.bf16_round(rng.standard_normal((n, m - k)).astype(np.float32)), layout))
    zf.scatter_weights(cols.t, sel, W.t, layout=layout)
    torch.cuda.synchronize()
    assert W.intact() and cols.intact()


@pytest.mark.parametrize("layout", LAYOUTS)
def test_no_write_outside_store_and_statistics(layout):
    """Swap-in / swap-out against a store and the Zen-auto statistics (plan
    path) write nothing outside their buffers."""
    n, m = 43, 77
    bits = grad_bits(n, m, 5)
    G = Guarded(*storage(layout, n, m), torch.bfloat16).fill(to_layout(bits, layout))
    rng = np.random.default_rng(3)
    old = O.select_topk(rng.random(m).astype(np.float32), 8)
    new = O.select_topk(rng.random(m).astype(np.float32), 8)

    def dev_sel(s):
        out = zf.Selection(s.m, s.k)
        out.sel_idx.copy_(torch.from_numpy(s.sel.astype(np.int32)))
        out.unsel_idx.copy_(torch.from_numpy(s.unsel.astype(np.int32)))
        out.mask.copy_(torch.from_numpy(s.mask.view(np.int64)))
        out.prefix.copy_(torch.from_numpy(s.prefix.astype(np.int32)))
        return out

    store = [Guarded(*storage(layout, n, m), torch.float32).fill(
        to_layout(rng.standard_normal((n, m)).astype(np.float32), layout)) for _ in range(3)]
    prev = [torch.from_numpy(to_layout(rng.standard_normal((n, 8)).astype(np.float32), layout))
            .cuda() for _ in range(3)]
    P, M, V = (Guarded(*storage(layout, n, 8), torch.float32) for _ in range(3))
    W = Guarded(*storage(layout, n, m), torch.bfloat16).fill(
        to_layout(np.zeros((n, m), np.uint16), layout))
    src = zf.StateSource(prev=dev_sel(old), prev_master=prev[0], prev_exp_avg=prev[1],
                         prev_exp_avg_sq=prev[2], store_master=store[0].t,
                         store_exp_avg=store[1].t, store_exp_avg_sq=store[2].t)
    zf.adam_selected(G.t, dev_sel(new), P.t, M.t, V.t, W.t, HP, 2, mode=zf.STATES_REMAP,
                     src=src, layout=layout)
    torch.cuda.synchronize()
    for g in store + [P, M, V, W]:
        assert g.intact()
    sel = dev_sel(new)
    k = sel.k
    A = Guarded(*storage(layout, n, m - k), torch.float32)
    ssq, asq = Guarded(1, k, torch.float32), Guarded(1, m - k, torch.float32)
    plan = zf.Plan([zf.MatrixBuffers(grad=G.t, k=k, sel=sel, weight=W.t, master=P.t,
                                     exp_avg=M.t, exp_avg_sq=V.t, acc=A.t, layout=layout,
                                     sel_sq=ssq.t.view(k), acc_sq=asq.t.view(m - k))])
    totals = torch.zeros(5, dtype=torch.int64, device="cuda")
    plan.update_zen(HP, 3, zf.STATES_INPLACE, 1, 4, 1.0, totals)
    torch.cuda.synchronize()
    for g in (A, ssq, asq, P, M, V, W):
        assert g.intact()
    assert ssq.fully_written() and asq.fully_written()
    plan.close()


@pytest.mark.parametrize("n,m", [(3, 7), (43, 77), (64, 130), (4104, 70), (16, 1000)])
@pytest.mark.parametrize("padded", [True, False], ids=["earlier-16B", "earlier-ld-eq-width"])
@pytest.mark.parametrize("layout", LAYOUTS)
def test_no_write_outside_deferred_handover(n, m, padded, layout):
    """zf_plan_update_handover_deferred (the interval's last step with
    deferred packing; three earlier gradients) writes nothing outside the
    compact states, W and the hand-over, fills the hand-over, leaves the
    earlier gradients alone, and equals the oracle: Adam in place on the
    selected columns, the hand-over of pack_accumulate over the four
    gradients times fp32(1/4).  Earlier gradients with 16-byte rows keep
    the row-major 16-byte kernel; unpadded ones (ld = width) take the
    per-column passes."""
    ratio = 0.1
    k = zf.k_from_ratio(ratio, m)
    rng = np.random.default_rng(n * 1000 + m)
    sel_h = O.select_topk(rng.random(m).astype(np.float32), k)
    sel = zf.Selection(m, k)
    sel.sel_idx.copy_(torch.from_numpy(sel_h.sel.astype(np.int32)))
    sel.unsel_idx.copy_(torch.from_numpy(sel_h.unsel.astype(np.int32)))
    sel.mask.copy_(torch.from_numpy(sel_h.mask.view(np.int64)))
    sel.prefix.copy_(torch.from_numpy(sel_h.prefix.astype(np.int32)))
    bits = [grad_bits(n, m, derive_seed("canary-deferred", n, m, s)) for s in range(4)]
    G = Guarded(*storage(layout, n, m), torch.bfloat16).fill(to_layout(bits[3], layout))
    if padded:
        E = [Guarded(*storage(layout, n, m), torch.bfloat16).fill(to_layout(b, layout))
             for b in bits[:3]]
        earlier_t = [e.t for e in E]
    else:
        E = []
        earlier_t = [torch.from_numpy(to_layout(b, layout).view(np.int16)).view(torch.bfloat16)
                     .cuda() for b in bits[:3]]
    before = [e.clone() for e in earlier_t]
    P0, M0 = (rng.standard_normal((n, k)).astype(np.float32) * 0.02 for _ in range(2))
    V0 = np.abs(rng.standard_normal((n, k)).astype(np.float32)) * 1e-4
    W0 = O.bf16_round((rng.standard_normal((n, m)) * 0.02).astype(np.float32))
    P, M, V = (Guarded(*storage(layout, n, k), torch.float32).fill(to_layout(x, layout))
               for x in (P0, M0, V0))
    W = Guarded(*storage(layout, n, m), torch.bfloat16).fill(to_layout(W0, layout))
    D = Guarded(*storage(layout, n, m), torch.float32)

    def buffers(grad):
        return zf.MatrixBuffers(grad=grad, k=k, sel=sel, weight=W.t, master=P.t, exp_avg=M.t,
                                exp_avg_sq=V.t, unpacked=D.t, layout=layout)
    plan = zf.Plan([buffers(G.t)])
    earlier = [zf.Plan([buffers(e)]) for e in earlier_t]
    step = 7
    plan.update_handover_deferred(HP, step, earlier, 0.25)
    torch.cuda.synchronize()
    for g in [P, M, V, W, D, G] + E:
        assert g.intact()
    assert D.fully_written()
    for a, b in zip(before, earlier_t):
        assert torch.equal(a.view(torch.int16), b.view(torch.int16))
    # against the oracle
    c = O.AdamConsts.at_step(HP.lr, HP.beta1, HP.beta2, HP.eps, HP.weight_decay, step)
    Pw, Mw, Vw, wsel = O.adam_selected(bits[3], sel_h.sel, P0, M0, V0, c)
    Ww = W0.copy()
    Ww[:, sel_h.sel.astype(np.int64)] = wsel
    A = None
    for s in range(4):
        A = O.pack_accumulate(bits[s], sel_h.unsel, A, s + 1)
    Dw = O.unpack(A, sel_h, float(np.float32(0.25)))

    def logical(t):
        x = t.t() if layout == zf.CHANNEL_MAJOR else t
        return x.contiguous().cpu()
    for got, want in ((P, Pw), (M, Mw), (V, Vw), (D, Dw)):
        assert np.array_equal(logical(got.t).view(torch.int32).numpy(),
                              np.ascontiguousarray(want, np.float32).view(np.int32))
    assert np.array_equal(logical(W.t).view(torch.int16).numpy().view(np.uint16), Ww)
    for e in earlier:
        e.close()
    plan.close()
