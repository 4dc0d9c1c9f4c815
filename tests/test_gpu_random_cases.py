"""Seeded random parity sweep through the C ABI: shapes, ratios, layouts and
buffer alignment drawn per case (so that every kernel variant -- the
channel-major update, the row-major 16-byte update and the row-major
per-column update -- meets ragged sizes it was not hand-picked for), each
case a short sequence checked against the oracle bit for bit:

  scores (1e-5 relative) -> top-k selection (bit-exact) -> init + pack ->
  in place + accumulate -> remap to the selection of new scores + pack ->
  fused hand-over.
"""
import numpy as np
import pytest
import torch

import oracle as O
from tests._gpu import bf16_dev, bits_np, f32_np, mask_np, rel_close, same_bits
from workloads import derive_seed, gradient

pytestmark = pytest.mark.gpu

zf = pytest.importorskip("paper_2505_12242_amd")
NCASES = 48


def case(seed):
    rng = np.random.default_rng(derive_seed("random-case", seed))
    n = int(rng.choice([1, 2, 3, 7, 16, 33, 64, 100, 257]))
    m = int(rng.choice([1, 5, 8, 63, 64, 65, 300, 999, 1000, 1001, 1500, 2048, 2999]))
    ratio = float(rng.choice([0.0, 1.0, rng.uniform(0.01, 0.6)]))
    layout = zf.ROW_MAJOR if rng.random() < 0.5 else zf.CHANNEL_MAJOR
    aligned = bool(rng.random() < 0.6)
    wd = float(rng.choice([0.0, 0.01]))
    return n, m, ratio, layout, aligned, wd, rng


class Bufs:
    """Device storage in `layout`, 16-byte aligned rows padded to 16 bytes,
    or a 4-byte (2-byte for bf16) offset with unpadded rows."""

    def __init__(self, layout, aligned):
        self.layout, self.aligned = layout, aligned

    def _shape(self, rows_l, cols_l):
        return (rows_l, cols_l) if self.layout == zf.ROW_MAJOR else (cols_l, rows_l)

    def f32(self, a):
        a = np.ascontiguousarray(a if self.layout == zf.ROW_MAJOR else np.asarray(a).T,
                                 dtype=np.float32)
        r, w = a.shape
        if self.aligned:
            per = 4
            ld = max(per, -(-w // per) * per)
            t = torch.empty(r, ld, device="cuda")[:, :w]
        else:
            t = torch.empty(r * w + 1, device="cuda")[1:].view(r, w)
        t.copy_(torch.from_numpy(a))
        return t

    def bf16(self, bits):
        b = bits if self.layout == zf.ROW_MAJOR else np.ascontiguousarray(bits.T)
        r, w = b.shape
        if self.aligned:
            return bf16_dev(b, ld=max(8, -(-w // 8) * 8))
        return bf16_dev(b, offset=1)

    def logical(self, t):
        a = f32_np(t) if t.dtype == torch.float32 else bits_np(t)
        return a if self.layout == zf.ROW_MAJOR else np.ascontiguousarray(a.T)


def grad_bits(n, m, seed):
    g = torch.Generator().manual_seed(seed)
    s = torch.exp(1.5 * torch.randn(m, generator=g, dtype=torch.float64))
    return bits_np(gradient(n, m, s, seed=seed))


@pytest.mark.parametrize("seed", range(NCASES))
def test_random_sequence(seed):
    n, m, ratio, layout, aligned, wd, rng = case(seed)
    hp = zf.AdamHparams(lr=1e-3, weight_decay=wd)
    consts = lambda t: O.AdamConsts.at_step(hp.lr, hp.beta1, hp.beta2, hp.eps, wd, t)
    B = Bufs(layout, aligned)
    k = zf.k_from_ratio(ratio, m)
    u = m - k
    W = O.bf16_round((rng.standard_normal((n, m)) * 0.02).astype(np.float32))
    Wd = B.bf16(W)
    tag = (seed, n, m, ratio, "rm" if layout == zf.ROW_MAJOR else "cm", aligned)

    # step 1: scores, selection, init + pack (overwrite)
    g1 = grad_bits(n, m, derive_seed("random-g", seed, 1))
    G1 = B.bf16(g1)
    s1 = zf.colnorm(G1, layout=layout)
    sel1 = zf.topk_select(s1, ratio)
    torch.cuda.synchronize()
    ok, worst = rel_close(f32_np(s1), O.colnorm(g1), 1e-5)
    assert ok, (tag, worst)
    o1 = O.select_topk(f32_np(s1), k)  # the oracle's selection of the device scores
    assert np.array_equal(sel1.sel_idx.cpu().numpy(), o1.sel), tag
    assert np.array_equal(sel1.unsel_idx.cpu().numpy(), o1.unsel), tag
    assert np.array_equal(mask_np(sel1.mask), o1.mask), tag
    P1, M1, V1 = (B.f32(np.full((n, k), np.nan, np.float32)) for _ in range(3))
    A = B.f32(np.full((n, u), np.nan, np.float32))
    zf.update_fused(G1, sel1, P1, M1, V1, Wd, hp, 1, A, 1, 3, mode=zf.STATES_INIT,
                    layout=layout)
    torch.cuda.synchronize()
    Pw, Mw, Vw = O.remap(None, o1, None, None, None, W, None)
    Pw, Mw, Vw, wsel = O.adam_selected(g1, o1.sel, Pw, Mw, Vw, consts(1))
    W[:, o1.sel.astype(np.int64)] = wsel
    Aw = O.pack_accumulate(g1, o1.unsel, None, 1)
    for got, want in ((P1, Pw), (M1, Mw), (V1, Vw), (A, Aw)):
        assert same_bits(B.logical(got), want), (tag, 1)
    assert np.array_equal(B.logical(Wd), W), (tag, 1)

    # step 2: in place + accumulate
    g2 = grad_bits(n, m, derive_seed("random-g", seed, 2))
    zf.update_fused(B.bf16(g2), sel1, P1, M1, V1, Wd, hp, 2, A, 2, 3, layout=layout)
    torch.cuda.synchronize()
    Pw, Mw, Vw, wsel = O.adam_selected(g2, o1.sel, Pw, Mw, Vw, consts(2))
    W[:, o1.sel.astype(np.int64)] = wsel
    Aw = O.pack_accumulate(g2, o1.unsel, Aw, 2)
    for got, want in ((P1, Pw), (M1, Mw), (V1, Vw), (A, Aw)):
        assert same_bits(B.logical(got), want), (tag, 2)
    assert np.array_equal(B.logical(Wd), W), (tag, 2)

    # step 3: new scores, remap + pack (overwrite)
    g3 = grad_bits(n, m, derive_seed("random-g", seed, 3))
    G3 = B.bf16(g3)
    s3 = zf.colnorm(G3, layout=layout)
    sel3 = zf.topk_select(s3, ratio)
    P3, M3, V3 = (B.f32(np.full((n, k), np.nan, np.float32)) for _ in range(3))
    src = zf.StateSource(prev=sel1, prev_master=P1, prev_exp_avg=M1, prev_exp_avg_sq=V1)
    zf.update_fused(G3, sel3, P3, M3, V3, Wd, hp, 3, A, 1, 3, mode=zf.STATES_REMAP, src=src,
                    layout=layout)
    torch.cuda.synchronize()
    o3 = O.select_topk(f32_np(s3), k)
    assert np.array_equal(sel3.sel_idx.cpu().numpy(), o3.sel), tag
    Pr, Mr, Vr = O.remap(o1, o3, Pw, Mw, Vw, W, None)
    Pw, Mw, Vw, wsel = O.adam_selected(g3, o3.sel, Pr, Mr, Vr, consts(3))
    W[:, o3.sel.astype(np.int64)] = wsel
    Aw = O.pack_accumulate(g3, o3.unsel, None, 1)
    for got, want in ((P3, Pw), (M3, Mw), (V3, Vw), (A, Aw)):
        assert same_bits(B.logical(got), want), (tag, 3)
    assert np.array_equal(B.logical(Wd), W), (tag, 3)

    # step 4: fused hand-over of a two-step interval (A only read)
    g4 = grad_bits(n, m, derive_seed("random-g", seed, 4))
    D = B.f32(np.full((n, m), np.nan, np.float32))
    scale = float(np.float32(0.5))
    zf.update_fused_handover(B.bf16(g4), sel3, P3, M3, V3, Wd, hp, 4, A, 2, 2, scale, out=D,
                             layout=layout)
    torch.cuda.synchronize()
    Pw, Mw, Vw, wsel = O.adam_selected(g4, o3.sel, Pw, Mw, Vw, consts(4))
    W[:, o3.sel.astype(np.int64)] = wsel
    Dw = O.unpack(O.pack_accumulate(g4, o3.unsel, Aw, 2), o3, scale)
    for got, want in ((P3, Pw), (M3, Mw), (V3, Vw), (A, Aw), (D, Dw)):
        assert same_bits(B.logical(got), want), (tag, 4)
    assert np.array_equal(B.logical(Wd), W), (tag, 4)
