"""Row-major update with 16-byte accesses: the kernel the library runs for
steps with the compact states in place (and pack-only calls) when G rows are
16-byte aligned (row stride a multiple of 8 bf16) and the packed buffer, the
compact states and the hand-over rows are 16-byte aligned with row strides
that are multiples of 4 floats; refresh steps and other buffers take the
per-column kernel.  Parity with the oracle bit for bit (states, weights,
packed buffer, hand-over) over

* tile raggedness: widths below, at and above the 1000-column tile limit,
  partial slot quads at both ends of each tile's unselected range, ratios 0
  and 1, row counts that leave a partial batch of rows;
* sequences that alternate the two kernels: init from W or from an fp32
  master, in place, a remap to a new selection, the fused hand-over; a
  refresh against a full-state store followed by in-place steps;
* pack-only and Adam-only calls, the fused update and the fused hand-over;
* the same sequences in unaligned buffers (per-column kernel throughout):
  identical bits.
"""
import numpy as np
import pytest
import torch

import oracle as O
from tests._gpu import bf16_dev, bits_np, f32_np, same_bits
from workloads import derive_seed, gradient

pytestmark = pytest.mark.gpu

zf = pytest.importorskip("paper_2505_12242_amd")
HP = zf.AdamHparams(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.01)
SHAPES = [(2, 8, 0.5), (3, 9, 0.34), (17, 77, 0.1), (5, 1008, 0.1), (20, 1009, 0.1),
          (9, 2017, 0.03), (16, 4096, 0.1), (37, 3000, 0.5), (5, 1500, 1.0), (6, 1500, 0.0),
          (33, 11008, 0.1), (70, 333, 0.25)]


def grad_bits(n, m, seed):
    g = torch.Generator().manual_seed(seed)
    s = torch.exp(1.5 * torch.randn(m, generator=g, dtype=torch.float64))
    return bits_np(gradient(n, m, s, seed=seed))


def consts(t):
    return O.AdamConsts.at_step(HP.lr, HP.beta1, HP.beta2, HP.eps, HP.weight_decay, t)


def sel_dev(s: O.Selection):
    out = zf.Selection(s.m, s.k)
    out.sel_idx.copy_(torch.from_numpy(s.sel.astype(np.int32)))
    out.unsel_idx.copy_(torch.from_numpy(s.unsel.astype(np.int32)))
    out.mask.copy_(torch.from_numpy(s.mask.view(np.int64)))
    out.prefix.copy_(torch.from_numpy(s.prefix.astype(np.int32)))
    return out


class Bufs:
    """Row-major fp32 / bf16 device buffers, aligned for the 16-byte path or
    deliberately misaligned (first element 4 or 2 bytes past a 16-byte
    boundary) for the per-column path."""

    def __init__(self, aligned: bool):
        self.aligned = aligned

    def f32(self, a):
        a = np.ascontiguousarray(a, dtype=np.float32)
        n, w = a.shape
        if self.aligned:
            t = zf.alloc_stored(zf.ROW_MAJOR, n, w)
        else:
            t = torch.empty(n * w + 1, device="cuda")[1:].view(n, w)
        t.copy_(torch.from_numpy(a))
        return t

    def nan(self, n, w):
        return self.f32(np.full((n, w), np.nan, np.float32))

    def bf16(self, bits):
        n, m = bits.shape
        if self.aligned:
            return bf16_dev(bits, ld=-(-m // 8) * 8)
        return bf16_dev(bits, offset=1)


def check(P, M, V, Pw, Mw, Vw, tag):
    assert same_bits(f32_np(P), Pw), (tag, "P")
    assert same_bits(f32_np(M), Mw), (tag, "M")
    assert same_bits(f32_np(V), Vw), (tag, "V")


def run_sequence(n, m, ratio, aligned, use_master):
    """INIT (fused, first step of an interval) -> in place (fused,
    accumulate) -> REMAP to a new selection (fused, first step) -> fused
    hand-over; each step checked against the oracle.  Returns the device
    results of every step for cross-path comparison."""
    B = Bufs(aligned)
    rng = np.random.default_rng(derive_seed("rv-seq", n, m))
    k = O.k_from_ratio(ratio, m)
    sel1 = O.select_topk(rng.random(m).astype(np.float32), k)
    sel2 = O.select_topk(rng.random(m).astype(np.float32), k)
    W = O.bf16_round((rng.standard_normal((n, m)) * 0.02).astype(np.float32))
    master = (rng.standard_normal((n, m)) * 0.02).astype(np.float32)
    Wd = B.bf16(W)
    out = []

    # step 1: INIT + pack (overwrite)
    g1 = grad_bits(n, m, derive_seed("rv-g", n, m, 1))
    P1, M1, V1 = (B.nan(n, k) for _ in range(3))
    A = B.nan(n, m - k)
    src = zf.StateSource(init_master=B.f32(master)) if use_master else None
    zf.update_fused(B.bf16(g1), sel_dev(sel1), P1, M1, V1, Wd, HP, 1, A, 1, 4,
                    mode=zf.STATES_INIT, src=src)
    torch.cuda.synchronize()
    Pw, Mw, Vw = O.remap(None, sel1, None, None, None, W, master if use_master else None)
    Pw, Mw, Vw, wsel = O.adam_selected(g1, sel1.sel, Pw, Mw, Vw, consts(1))
    W[:, sel1.sel.astype(np.int64)] = wsel
    Aw = O.pack_accumulate(g1, sel1.unsel, None, 1)
    check(P1, M1, V1, Pw, Mw, Vw, "init")
    assert np.array_equal(bits_np(Wd), W), "init W"
    assert same_bits(f32_np(A), Aw), "init A"
    out.append([f32_np(x) for x in (P1, M1, V1, A)] + [bits_np(Wd)])

    # step 2: in place + accumulate
    g2 = grad_bits(n, m, derive_seed("rv-g", n, m, 2))
    zf.update_fused(B.bf16(g2), sel_dev(sel1), P1, M1, V1, Wd, HP, 2, A, 2, 4)
    torch.cuda.synchronize()
    Pw, Mw, Vw, wsel = O.adam_selected(g2, sel1.sel, Pw, Mw, Vw, consts(2))
    W[:, sel1.sel.astype(np.int64)] = wsel
    Aw = O.pack_accumulate(g2, sel1.unsel, Aw, 2)
    check(P1, M1, V1, Pw, Mw, Vw, "inplace")
    assert np.array_equal(bits_np(Wd), W), "inplace W"
    assert same_bits(f32_np(A), Aw), "inplace A"
    out.append([f32_np(x) for x in (P1, M1, V1, A)] + [bits_np(Wd)])

    # step 3: refresh -> REMAP to sel2, new interval (overwrite)
    g3 = grad_bits(n, m, derive_seed("rv-g", n, m, 3))
    P2, M2, V2 = (B.nan(n, k) for _ in range(3))
    src = zf.StateSource(prev=sel_dev(sel1), prev_master=P1, prev_exp_avg=M1, prev_exp_avg_sq=V1,
                         init_master=B.f32(master) if use_master else None)
    zf.update_fused(B.bf16(g3), sel_dev(sel2), P2, M2, V2, Wd, HP, 3, A, 1, 4,
                    mode=zf.STATES_REMAP, src=src)
    torch.cuda.synchronize()
    Pr, Mr, Vr = O.remap(sel1, sel2, Pw, Mw, Vw, W, master if use_master else None)
    Pw, Mw, Vw, wsel = O.adam_selected(g3, sel2.sel, Pr, Mr, Vr, consts(3))
    W[:, sel2.sel.astype(np.int64)] = wsel
    Aw = O.pack_accumulate(g3, sel2.unsel, None, 1)
    check(P2, M2, V2, Pw, Mw, Vw, "remap")
    assert np.array_equal(bits_np(Wd), W), "remap W"
    assert same_bits(f32_np(A), Aw), "remap A"
    out.append([f32_np(x) for x in (P2, M2, V2, A)] + [bits_np(Wd)])

    # step 4: fused hand-over (A only read)
    g4 = grad_bits(n, m, derive_seed("rv-g", n, m, 4))
    D = B.nan(n, m)
    scale = float(np.float32(0.5))
    zf.update_fused_handover(B.bf16(g4), sel_dev(sel2), P2, M2, V2, Wd, HP, 4, A, 2, 2, scale,
                             out=D)
    torch.cuda.synchronize()
    Pw, Mw, Vw, wsel = O.adam_selected(g4, sel2.sel, Pw, Mw, Vw, consts(4))
    W[:, sel2.sel.astype(np.int64)] = wsel
    Dw = O.unpack(O.pack_accumulate(g4, sel2.unsel, Aw, 2), sel2, scale)
    check(P2, M2, V2, Pw, Mw, Vw, "handover")
    assert np.array_equal(bits_np(Wd), W), "handover W"
    assert same_bits(f32_np(A), Aw), "handover leaves A"
    assert same_bits(f32_np(D), Dw), "handover D"
    out.append([f32_np(x) for x in (P2, M2, V2, D)] + [bits_np(Wd)])
    return out


@pytest.mark.parametrize("n,m,ratio", SHAPES)
@pytest.mark.parametrize("use_master", [False, True])
def test_sequence_matches_oracle_and_per_column_path(n, m, ratio, use_master):
    vec = run_sequence(n, m, ratio, True, use_master)
    col = run_sequence(n, m, ratio, False, use_master)
    for s, (a, b) in enumerate(zip(vec, col)):
        for x, y in zip(a, b):
            assert same_bits(x, y), s


@pytest.mark.parametrize("n,m,ratio", [(17, 77, 0.1), (20, 1009, 0.1), (33, 11008, 0.1),
                                       (9, 2017, 0.5), (5, 40, 1.0), (6, 40, 0.0)])
def test_pack_only_and_adam_only(n, m, ratio):
    B = Bufs(True)
    rng = np.random.default_rng(derive_seed("rv-split", n, m))
    sel = O.select_topk(rng.random(m).astype(np.float32), O.k_from_ratio(ratio, m))
    k = sel.k
    P = (rng.standard_normal((n, k)) * 0.02).astype(np.float32)
    M = (rng.standard_normal((n, k)) * 1e-3).astype(np.float32)
    V = (rng.random((n, k)) * 1e-4).astype(np.float32)
    W = O.bf16_round((rng.standard_normal((n, m)) * 0.02).astype(np.float32))
    Pd, Md, Vd, Wd = B.f32(P), B.f32(M), B.f32(V), B.bf16(W)
    A = B.nan(n, m - k)
    Aw = None
    for t in (1, 2, 3):
        g = grad_bits(n, m, derive_seed("rv-split-g", n, m, t))
        g[0, ::7] = 0x8000  # -0.0 survives the overwrite
        zf.pack_accumulate(B.bf16(g), sel_dev(sel), A, t, 3)
        zf.adam_selected(B.bf16(g), sel_dev(sel), Pd, Md, Vd, Wd, HP, t)
        torch.cuda.synchronize()
        Aw = O.pack_accumulate(g, sel.unsel, Aw, t)
        P, M, V, wsel = O.adam_selected(g, sel.sel, P, M, V, consts(t))
        W[:, sel.sel.astype(np.int64)] = wsel
        assert same_bits(f32_np(A), Aw), t
        check(Pd, Md, Vd, P, M, V, t)
        assert np.array_equal(bits_np(Wd), W), t


@pytest.mark.parametrize("n,m", [(33, 300), (8, 1009), (21, 4096), (5, 9)])
@pytest.mark.parametrize("where", ["device", "pinned"])
def test_swap_against_store(n, m, where):
    """Refresh with a full-state store: staying columns move to their new
    slot, entering columns swap in from the store, leaving columns swap out
    to it (the store in device memory or in pinned host memory); then
    in-place steps on the swapped-in states."""
    B = Bufs(True)
    rng = np.random.default_rng(derive_seed("rv-swap", n, m))
    bits = grad_bits(n, m, derive_seed("rv-swap-g", n, m))
    W = O.bf16_round((rng.standard_normal((n, m)) * 0.02).astype(np.float32))
    k_old, k_new = O.k_from_ratio(0.15, m), O.k_from_ratio(0.2, m)
    old = O.select_topk(rng.random(m).astype(np.float32), k_old)
    new = O.select_topk(rng.random(m).astype(np.float32), k_new)
    P = (rng.standard_normal((n, k_old)) * 0.02).astype(np.float32)
    M = (rng.standard_normal((n, k_old)) * 1e-3).astype(np.float32)
    V = np.abs(rng.standard_normal((n, k_old)) * 1e-5).astype(np.float32)
    store = ((rng.standard_normal((n, m)) * 0.02).astype(np.float32),
             (rng.standard_normal((n, m)) * 1e-3).astype(np.float32),
             (rng.random((n, m)) * 1e-5).astype(np.float32))
    if where == "device":
        sd = [B.f32(x) for x in store]
    else:
        sd = []
        for x in store:
            p = torch.empty(x.shape, dtype=torch.float32, pin_memory=True)
            p.copy_(torch.from_numpy(x))
            sd.append(p)
    Pn, Mn, Vn = (B.nan(n, k_new) for _ in range(3))
    A = B.nan(n, m - k_new)
    Wd = B.bf16(W)
    src = zf.StateSource(prev=sel_dev(old), prev_master=B.f32(P), prev_exp_avg=B.f32(M),
                         prev_exp_avg_sq=B.f32(V), store_master=sd[0], store_exp_avg=sd[1],
                         store_exp_avg_sq=sd[2])
    zf.update_fused(B.bf16(bits), sel_dev(new), Pn, Mn, Vn, Wd, HP, 5, A, 1, 4,
                    mode=zf.STATES_REMAP, src=src)
    torch.cuda.synchronize()
    P2, M2, V2, store2 = O.swap_states(old, new, P, M, V, store)
    Pw, Mw, Vw, wsel = O.adam_selected(bits, new.sel, P2, M2, V2, consts(5))
    check(Pn, Mn, Vn, Pw, Mw, Vw, "swap")
    Wwant = W.copy()
    Wwant[:, new.sel.astype(np.int64)] = wsel
    assert np.array_equal(bits_np(Wd), Wwant)
    for got, want in zip(sd, store2):
        assert same_bits(f32_np(got), want)
    Aw = O.pack_accumulate(bits, new.unsel, None, 1)
    assert same_bits(f32_np(A), Aw)
    # then in-place steps on the swapped-in states (16-byte kernel)
    for t, sii in ((6, 2), (7, 3)):
        g = grad_bits(n, m, derive_seed("rv-swap-g", n, m, t))
        zf.update_fused(B.bf16(g), sel_dev(new), Pn, Mn, Vn, Wd, HP, t, A, sii, 4)
        torch.cuda.synchronize()
        Pw, Mw, Vw, wsel = O.adam_selected(g, new.sel, Pw, Mw, Vw, consts(t))
        Wwant[:, new.sel.astype(np.int64)] = wsel
        Aw = O.pack_accumulate(g, new.unsel, Aw, sii)
        check(Pn, Mn, Vn, Pw, Mw, Vw, t)
        assert np.array_equal(bits_np(Wd), Wwant), t
        assert same_bits(f32_np(A), Aw), t


def test_plan_uses_padded_buffers():
    """A multi-matrix plan over padded buffers (16-byte path) equals the
    single-matrix calls over unaligned buffers (per-column path)."""
    shapes = [(40, 1009, 0.1), (17, 77, 0.25), (8, 4096, 0.05)]
    rng = np.random.default_rng(11)
    A_al, B_un = Bufs(True), Bufs(False)
    mats, twins = [], []
    for q, (n, m, ratio) in enumerate(shapes):
        sel = O.select_topk(rng.random(m).astype(np.float32), O.k_from_ratio(ratio, m))
        k = sel.k
        g = grad_bits(n, m, derive_seed("rv-plan", q))
        P = (rng.standard_normal((n, k)) * 0.02).astype(np.float32)
        M = (rng.standard_normal((n, k)) * 1e-3).astype(np.float32)
        V = (rng.random((n, k)) * 1e-4).astype(np.float32)
        W = O.bf16_round((rng.standard_normal((n, m)) * 0.02).astype(np.float32))
        Acc = rng.standard_normal((n, m - k)).astype(np.float32)
        bufs = dict(grad=A_al.bf16(g), weight=A_al.bf16(W), master=A_al.f32(P),
                    exp_avg=A_al.f32(M), exp_avg_sq=A_al.f32(V), acc=A_al.f32(Acc),
                    unpacked=A_al.nan(n, m))
        twin = dict(grad=B_un.bf16(g), weight=B_un.bf16(W), master=B_un.f32(P),
                    exp_avg=B_un.f32(M), exp_avg_sq=B_un.f32(V), acc=B_un.f32(Acc),
                    unpacked=B_un.nan(n, m))
        s = sel_dev(sel)
        mats.append(zf.MatrixBuffers(k=k, sel=s, layout=zf.ROW_MAJOR, **bufs))
        twins.append((s, twin))
    plan = zf.Plan(mats)
    plan.update(HP, 6, zf.STATES_INPLACE, 2, 4, True, True)
    plan.update_handover(HP, 7, zf.STATES_INPLACE, 3, 4, 0.25)
    for s, b in twins:
        zf.update_fused(b["grad"], s, b["master"], b["exp_avg"], b["exp_avg_sq"], b["weight"],
                        HP, 6, b["acc"], 2, 4)
        zf.update_fused_handover(b["grad"], s, b["master"], b["exp_avg"], b["exp_avg_sq"],
                                 b["weight"], HP, 7, b["acc"], 3, 4, 0.25, out=b["unpacked"])
    torch.cuda.synchronize()
    for mb, (s, b) in zip(mats, twins):
        for name in ("master", "exp_avg", "exp_avg_sq", "acc", "unpacked"):
            assert same_bits(f32_np(getattr(mb, name)), f32_np(b[name])), name
        assert np.array_equal(bits_np(mb.weight), bits_np(b["weight"]))
    plan.close()


@pytest.mark.parametrize("n,m,ratio", [(1, 77, 0.1), (2, 8, 0.5), (17, 1009, 0.1), (9, 2017, 0.0),
                                       (5, 300, 1.0)])
@pytest.mark.parametrize("aligned", [True, False])
def test_handover_on_first_step(n, m, ratio, aligned):
    """A one-step interval (warm-up, or a refresh every step) hands over on
    its first step: the packed buffer is neither read nor written and the
    hand-over is scale * the gradient at the unselected columns."""
    B = Bufs(aligned)
    rng = np.random.default_rng(derive_seed("rv-first", n, m))
    sel = O.select_topk(rng.random(m).astype(np.float32), O.k_from_ratio(ratio, m))
    k = sel.k
    P = (rng.standard_normal((n, k)) * 0.02).astype(np.float32)
    M = (rng.standard_normal((n, k)) * 1e-3).astype(np.float32)
    V = (rng.random((n, k)) * 1e-4).astype(np.float32)
    W = O.bf16_round((rng.standard_normal((n, m)) * 0.02).astype(np.float32))
    Pd, Md, Vd, Wd = B.f32(P), B.f32(M), B.f32(V), B.bf16(W)
    A = B.nan(n, m - k)
    D = B.nan(n, m)
    g = grad_bits(n, m, derive_seed("rv-first-g", n, m))
    g[0, ::5] = 0x8000  # -0.0 survives
    zf.update_fused_handover(B.bf16(g), sel_dev(sel), Pd, Md, Vd, Wd, HP, 9, A, 1, 1, 1.0,
                             out=D)
    torch.cuda.synchronize()
    Pw, Mw, Vw, wsel = O.adam_selected(g, sel.sel, P, M, V, consts(9))
    W[:, sel.sel.astype(np.int64)] = wsel
    check(Pd, Md, Vd, Pw, Mw, Vw, "first")
    assert np.array_equal(bits_np(Wd), W)
    assert np.isnan(f32_np(A)).all()  # not written
    assert same_bits(f32_np(D), O.unpack(O.pack_accumulate(g, sel.unsel, None, 1), sel, 1.0))
