"""Parity of each C-ABI entry point with the CPU oracle on seeded inputs:
ragged shapes, padded and unaligned strides, ties, empty and degenerate
sizes.  Bar: bit-exact indices, masks, prefixes, packed and unpacked
buffers; scores within 1e-5 relative; fp32 Adam states within 2e-6
relative (first moment floored at 2e-6 of its summands), bf16 weights
bit-exact wherever the master is."""
import numpy as np
import pytest
import torch

import oracle as O
from tests._gpu import (bf16_dev, bits_np, f32_dev, f32_np, mask_np, rel_close, same_bits)
from workloads import derive_seed, gradient, score_vector

pytestmark = pytest.mark.gpu

zf = pytest.importorskip("paper_2505_12242_amd")
HP = zf.AdamHparams(lr=1e-5, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.0)
LAYOUTS = [pytest.param(zf.ROW_MAJOR, id="rm"), pytest.param(zf.CHANNEL_MAJOR, id="cm")]


def T(a, layout):
    """Logical [rows][cols] host array -> its storage in `layout`."""
    return a if layout == zf.ROW_MAJOR else np.ascontiguousarray(np.asarray(a).T)


def bits_dev(bits, layout, **kw):
    return bf16_dev(T(bits, layout), **kw)


def f32_dev_l(a, layout):
    return f32_dev(T(a, layout))


def f32_host(t, layout):
    a = f32_np(t)
    return a if layout == zf.ROW_MAJOR else np.ascontiguousarray(a.T)


def bits_host(t, layout):
    b = bits_np(t)
    return b if layout == zf.ROW_MAJOR else np.ascontiguousarray(b.T)


def grad_bits(n, m, seed, sigma=1.5):
    g = torch.Generator().manual_seed(seed)
    s = torch.exp(sigma * torch.randn(m, generator=g, dtype=torch.float64))
    return bits_np(gradient(n, m, s, seed=seed))


def oracle_consts(hp, t):
    return O.AdamConsts.at_step(hp.lr, hp.beta1, hp.beta2, hp.eps, hp.weight_decay, t)


def sel_from_oracle(s: O.Selection):
    out = zf.Selection(s.m, s.k)
    out.sel_idx.copy_(torch.from_numpy(s.sel.astype(np.int32)))
    out.unsel_idx.copy_(torch.from_numpy(s.unsel.astype(np.int32)))
    out.mask.copy_(torch.from_numpy(s.mask.view(np.int64)))
    out.prefix.copy_(torch.from_numpy(s.prefix.astype(np.int32)))
    return out


# ---------------------------------------------------------------- colnorm

SHAPES = [(1, 1), (1, 513), (2, 3), (3, 7), (7, 8), (8, 63), (63, 64), (64, 65), (65, 513),
          (513, 100), (700, 4097), (4097, 65), (0, 9)]


@pytest.mark.parametrize("n,m", SHAPES)
@pytest.mark.parametrize("storage", ["dense", "padded", "offset"])
@pytest.mark.parametrize("layout", LAYOUTS)
def test_colnorm(n, m, storage, layout):
    bits = grad_bits(n, m, derive_seed("cn", n, m))
    bits[:, ::7] = 0  # zero columns must give exactly 0
    width = m if layout == zf.ROW_MAJOR else n
    if storage == "dense":
        G = bits_dev(bits, layout)
    elif storage == "padded":
        G = bits_dev(bits, layout, ld=((width + 7) // 8) * 8 + 8)
    else:
        G = bits_dev(bits, layout, ld=width + 3, offset=1)
    got = f32_np(zf.colnorm(G, layout=layout))
    torch.cuda.synchronize()
    want = O.colnorm(bits)
    ok, worst = rel_close(got, want, 1e-5)
    assert ok, worst
    assert np.all(got[want == 0] == 0)
    if n == 1:
        assert same_bits(got, want)


@pytest.mark.parametrize("layout", LAYOUTS)
def test_colnorm_exact_cases(layout):
    n, m = 300, 70
    bits = np.zeros((n, m), np.uint16)
    bits[:, 5] = 0x3E00  # 0.125 -> n/64 exactly
    bits[::3, 9] = 0xC100  # -8
    got = f32_np(zf.colnorm(bits_dev(bits, layout), layout=layout))
    assert got[5] == np.float32(n / 64) and got[9] == np.float32(100 * 64)
    assert np.count_nonzero(got) == 2


# ---------------------------------------------------------------- top-k

KINDS = ["lognormal", "wide", "ties", "few-distinct", "constant", "zeros", "signed-zero"]


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("m", [1, 5, 63, 64, 65, 1000, 4096, 11008, 28672, 70001])
def test_topk(kind, m):
    s = score_vector(m, seed=derive_seed("tk", kind, m), kind=kind).numpy()
    S = f32_dev(s)
    ratios = {0.0, 0.01, 0.1, 0.5, 1.0, (1 + 0.01) / m, (m - 1 + 0.01) / m}
    for ratio in sorted(r for r in ratios if 0 <= r <= 1):
        got = zf.topk_select(S, ratio)
        torch.cuda.synchronize()
        want = O.select_topk(s, O.k_from_ratio(ratio, m))
        assert got.k == want.k
        assert np.array_equal(got.sel_idx.cpu().numpy(), want.sel), (kind, m, ratio)
        assert np.array_equal(got.unsel_idx.cpu().numpy(), want.unsel), (kind, m, ratio)
        assert np.array_equal(mask_np(got.mask), want.mask), (kind, m, ratio)
        assert np.array_equal(got.prefix.cpu().numpy(), want.prefix), (kind, m, ratio)


# ---------------------------------------------------------------- Adam

def adam_case(n, m, ratio, seed):
    rng = np.random.default_rng(seed)
    bits = grad_bits(n, m, seed)
    scores = rng.random(m).astype(np.float32)
    sel = O.select_topk(scores, O.k_from_ratio(ratio, m))
    k = sel.k
    P = (rng.standard_normal((n, k)) * 0.02).astype(np.float32)
    M = (rng.standard_normal((n, k)) * 1e-3).astype(np.float32)
    V = (rng.random((n, k)) * 1e-4).astype(np.float32)
    W = O.bf16_round((rng.standard_normal((n, m)) * 0.02).astype(np.float32))
    return bits, sel, P, M, V, W


def check_states(P, M, V, Pw, Mw, Vw, g_abs, Mprev):
    ok, w = rel_close(P, Pw, 2e-6)
    assert ok, ("P", w)
    ok, w = rel_close(V, Vw, 2e-6)
    assert ok, ("V", w)
    ok, w = rel_close(M, Mw, 2e-6, floor=2e-6 * (0.9 * np.abs(Mprev) + 0.1 * g_abs))
    assert ok, ("M", w)


@pytest.mark.parametrize("n,m,ratio", [(1, 1, 1.0), (3, 7, 0.3), (64, 65, 0.1), (65, 513, 0.1),
                                       (513, 1000, 0.25), (130, 4097, 0.01), (7, 64, 1.0)])
@pytest.mark.parametrize("wd", [0.0, 0.01])
@pytest.mark.parametrize("step", [1, 7])
@pytest.mark.parametrize("layout", LAYOUTS)
def test_adam_inplace(n, m, ratio, wd, step, layout):
    bits, sel, P, M, V, W = adam_case(n, m, ratio, derive_seed("adam", n, m))
    hp = zf.AdamHparams(weight_decay=wd)
    Pd, Md, Vd, Wd = f32_dev_l(P, layout), f32_dev_l(M, layout), f32_dev_l(V, layout), \
        bits_dev(W, layout)
    ld = (m if layout == zf.ROW_MAJOR else n) + 5
    zf.adam_selected(bits_dev(bits, layout, ld=ld), sel_from_oracle(sel), Pd, Md, Vd, Wd, hp,
                     step, layout=layout)
    torch.cuda.synchronize()
    Pw, Mw, Vw, wsel = O.adam_selected(bits, sel.sel, P, M, V, oracle_consts(hp, step))
    g_abs = np.abs(O.widen(bits[:, sel.sel.astype(np.int64)]))
    Pg, Mg, Vg = f32_host(Pd, layout), f32_host(Md, layout), f32_host(Vd, layout)
    check_states(Pg, Mg, Vg, Pw, Mw, Vw, g_abs, M)
    Wgot = bits_host(Wd, layout)
    Wwant = W.copy()
    Wwant[:, sel.sel.astype(np.int64)] = wsel
    same = same_bits(Pg, Pw)
    if same:
        assert np.array_equal(Wgot, Wwant)
    else:
        diff = np.abs(Wgot.astype(np.int32) - Wwant.astype(np.int32))
        assert diff.max() <= 1
    # report exactness (the kernel is written to reproduce the oracle's rounding)
    assert same_bits(Mg, Mw) and same_bits(Vg, Vw) and same


@pytest.mark.parametrize("use_master", [False, True])
@pytest.mark.parametrize("layout", LAYOUTS)
def test_adam_remap_and_init(use_master, layout):
    n, m = 33, 300
    rng = np.random.default_rng(5)
    bits = grad_bits(n, m, 17)
    W = O.bf16_round((rng.standard_normal((n, m)) * 0.02).astype(np.float32))
    master = (rng.standard_normal((n, m)) * 0.02).astype(np.float32)
    old = O.select_topk(rng.random(m).astype(np.float32), 40)
    new = O.select_topk(rng.random(m).astype(np.float32), 45)
    P = (rng.standard_normal((n, 40)) * 0.02).astype(np.float32)
    M = (rng.standard_normal((n, 40)) * 1e-3).astype(np.float32)
    V = (rng.random((n, 40)) * 1e-4).astype(np.float32)
    old_d, new_d = sel_from_oracle(old), sel_from_oracle(new)
    shape = (n, 45) if layout == zf.ROW_MAJOR else (45, n)
    Pn = torch.full(shape, np.nan, device="cuda")
    Mn, Vn = torch.full_like(Pn, np.nan), torch.full_like(Pn, np.nan)
    Wd = bits_dev(W, layout)
    src = zf.StateSource(prev=old_d, prev_master=f32_dev_l(P, layout),
                         prev_exp_avg=f32_dev_l(M, layout), prev_exp_avg_sq=f32_dev_l(V, layout),
                         init_master=f32_dev_l(master, layout) if use_master else None)
    zf.adam_selected(bits_dev(bits, layout), new_d, Pn, Mn, Vn, Wd, HP, 3, mode=zf.STATES_REMAP,
                     src=src, layout=layout)
    torch.cuda.synchronize()
    P2, M2, V2 = O.remap(old, new, P, M, V, W, master if use_master else None)
    Pw, Mw, Vw, wsel = O.adam_selected(bits, new.sel, P2, M2, V2, oracle_consts(HP, 3))
    assert same_bits(f32_host(Pn, layout), Pw) and same_bits(f32_host(Mn, layout), Mw)
    assert same_bits(f32_host(Vn, layout), Vw)
    assert np.array_equal(bits_host(Wd, layout)[:, new.sel.astype(np.int64)], wsel)
    # INIT: every selected column starts fresh
    Pi, Mi, Vi = (torch.zeros(shape, device="cuda") for _ in range(3))
    Wd2 = bits_dev(W, layout)
    zf.adam_selected(bits_dev(bits, layout), new_d, Pi, Mi, Vi, Wd2, HP, 1, mode=zf.STATES_INIT,
                     src=zf.StateSource(init_master=f32_dev_l(master, layout) if use_master
                                        else None), layout=layout)
    torch.cuda.synchronize()
    P3, M3, V3 = O.remap(None, new, None, None, None, W, master if use_master else None)
    Pw, Mw, Vw, _ = O.adam_selected(bits, new.sel, P3, M3, V3, oracle_consts(HP, 1))
    assert same_bits(f32_host(Pi, layout), Pw) and same_bits(f32_host(Mi, layout), Mw)
    assert same_bits(f32_host(Vi, layout), Vw)


# ---------------------------------------------------------------- pack / unpack / fused

@pytest.mark.parametrize("n,m,ratio", [(1, 1, 0.0), (2, 3, 0.34), (65, 513, 0.1),
                                       (300, 4097, 0.05), (17, 64, 1.0), (9, 700, 0.0),
                                       (4104, 40, 0.1), (8200, 3, 0.34)])
@pytest.mark.parametrize("layout", LAYOUTS)
def test_pack_accumulate_and_unpack(n, m, ratio, layout):
    rng = np.random.default_rng(n * 1000 + m)
    sel = O.select_topk(rng.random(m).astype(np.float32), O.k_from_ratio(ratio, m))
    sd = sel_from_oracle(sel)
    u = m - sel.k
    S = 4
    rows, width = (n, u) if layout == zf.ROW_MAJOR else (u, n)
    A = torch.full((rows, width + 4), np.nan, device="cuda")[:, :width]  # padded, junk content
    Aw = None
    for t in range(1, S + 1):
        bits = grad_bits(n, m, derive_seed("pack", n, m, t))
        bits[0, ::5] = 0x8000  # -0.0 survives the overwrite
        zf.pack_accumulate(bits_dev(bits, layout), sd, A, t, S, layout=layout)
        Aw = O.pack_accumulate(bits, sel.unsel, Aw, t)
        torch.cuda.synchronize()
        assert same_bits(f32_host(A, layout), Aw), t
    drows, dwidth = (n, m) if layout == zf.ROW_MAJOR else (m, n)
    for scale in (1.0, 0.25, 1.0 / 3.0):
        D = torch.full((drows, dwidth + 4), 7.0, device="cuda")[:, :dwidth]
        zf.unpack(A, sd, scale, out=D, layout=layout)
        torch.cuda.synchronize()
        assert same_bits(f32_host(D, layout), O.unpack(Aw, sel, float(np.float32(scale))))


@pytest.mark.parametrize("n,m,ratio", [(65, 513, 0.1), (200, 4096, 0.1), (5, 9, 0.5),
                                       (4104, 70, 0.1)])
@pytest.mark.parametrize("layout", LAYOUTS)
def test_fused_equals_separate(n, m, ratio, layout):
    bits, sel, P, M, V, W = adam_case(n, m, ratio, derive_seed("fused", n, m))
    sd = sel_from_oracle(sel)
    G = bits_dev(bits, layout)
    L = layout
    a = [f32_dev_l(P, L), f32_dev_l(M, L), f32_dev_l(V, L), bits_dev(W, L)]
    b = [f32_dev_l(P, L), f32_dev_l(M, L), f32_dev_l(V, L), bits_dev(W, L)]
    ashape = (n, m - sel.k) if L == zf.ROW_MAJOR else (m - sel.k, n)
    A1 = torch.zeros(ashape, device="cuda")
    A2 = torch.zeros(ashape, device="cuda")
    zf.update_fused(G, sd, *a, HP, 2, A1, 1, 4, layout=L)
    zf.update_fused(G, sd, *a, HP, 3, A1, 2, 4, layout=L)
    for step, sii in ((2, 1), (3, 2)):
        zf.adam_selected(G, sd, *b, HP, step, layout=L)
        zf.pack_accumulate(G, sd, A2, sii, 4, layout=L)
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        assert torch.equal(x.view(torch.int32) if x.dtype == torch.float32 else x.view(torch.int16),
                           y.view(torch.int32) if y.dtype == torch.float32 else y.view(torch.int16))
    assert torch.equal(A1.view(torch.int32), A2.view(torch.int32))


@pytest.mark.parametrize("n,m,ratio", [(65, 513, 0.1), (200, 4096, 0.1), (5, 9, 0.5),
                                       (4104, 70, 0.1), (43, 77, 0.2), (16, 3, 0.1), (8, 10, 1.0)])
@pytest.mark.parametrize("sii", [1, 3])
@pytest.mark.parametrize("layout", LAYOUTS)
def test_fused_handover_equals_update_then_unpack(n, m, ratio, sii, layout):
    """The interval's last step in one pass (zf_update_fused_handover) equals
    zf_update_fused followed by zf_unpack bit for bit -- states, weights and
    the hand-over -- and leaves the packed buffer untouched."""
    bits, sel, P, M, V, W = adam_case(n, m, ratio, derive_seed("handover", n, m, sii))
    sd = sel_from_oracle(sel)
    G = bits_dev(bits, layout)
    L = layout
    a = [f32_dev_l(P, L), f32_dev_l(M, L), f32_dev_l(V, L), bits_dev(W, L)]
    b = [f32_dev_l(P, L), f32_dev_l(M, L), f32_dev_l(V, L), bits_dev(W, L)]
    u = m - sel.k
    rng = np.random.default_rng(n + m + sii)
    A0 = T(rng.standard_normal((n, u)).astype(np.float32), L)
    A1, A2 = f32_dev(A0), f32_dev(A0)
    scale = float(np.float32(1.0 / 3.0))
    oshape = (n, m) if L == zf.ROW_MAJOR else (m, n)
    D1 = torch.full((oshape[0], oshape[1] + 4), np.nan, device="cuda")[:, :oshape[1]]  # padded
    zf.update_fused_handover(G, sd, *a, HP, 7, A1, sii, 4, scale, out=D1, layout=L)
    zf.update_fused(G, sd, *b, HP, 7, A2, sii, 4, layout=L)
    D2 = zf.unpack(A2, sd, scale, layout=L)
    torch.cuda.synchronize()
    for x, y in zip(a, b):
        assert torch.equal(x.view(torch.int32) if x.dtype == torch.float32 else x.view(torch.int16),
                           y.view(torch.int32) if y.dtype == torch.float32 else y.view(torch.int16))
    assert same_bits(f32_np(D1), f32_np(D2))
    assert same_bits(f32_np(A1), A0)  # only read
    # and against the oracle's definition
    A_or = O.pack_accumulate(bits, sel.unsel, T(A0, L), sii)
    assert same_bits(f32_host(D1, L), O.unpack(A_or, sel, scale))


def test_empty_sizes_are_no_ops():
    G = torch.empty(0, 9, dtype=torch.bfloat16, device="cuda")
    s = zf.colnorm(G)
    s_cm = zf.colnorm(torch.empty(9, 0, dtype=torch.bfloat16, device="cuda"),
                      layout=zf.CHANNEL_MAJOR)
    torch.cuda.synchronize()
    assert torch.equal(s, torch.zeros(9, device="cuda"))
    assert torch.equal(s_cm, torch.zeros(9, device="cuda"))
    sel = zf.topk_select(torch.empty(0, device="cuda"), 0.1)
    assert sel.k == 0
    sd = zf.topk_select(torch.rand(9, device="cuda"), 0.5)
    zf.pack_accumulate(G, sd, torch.empty(0, 9 - sd.k, device="cuda"), 1, 1)
    torch.cuda.synchronize()


@pytest.mark.parametrize("layout", LAYOUTS)
def test_deterministic_reruns(layout):
    n, m = 2000, 3000
    G = bits_dev(grad_bits(n, m, 99), layout)
    a = zf.colnorm(G, layout=layout)
    b = zf.colnorm(G, layout=layout)
    sa = zf.topk_select(a, 0.1)
    sb = zf.topk_select(b, 0.1)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int32), b.view(torch.int32))
    assert torch.equal(sa.sel_idx, sb.sel_idx) and torch.equal(sa.mask, sb.mask)
