"""Deferred packing: the unselected part of each step's gradient stays in
its gradient slot and the interval's last step sums the interval's
gradients, in step order, into the hand-over
(zf_plan_update_handover_deferred); the other steps run Adam alone.  Three
storage variants: channel-major; row-major with 16-byte gradient rows (the
16-byte update kernel with the sum fused in, ragged tile ends included);
row-major with unpadded rows whose widths are not multiples of 8 (the
per-column Adam pass and the per-column hand-over pass).

* the runner in this mode against the oracle (MatrixOracle), every step:
  compact states and W bit for bit, selections bit-exact, the hand-over bit
  for bit at every interval end; schedules with refreshes that cut intervals
  short, one-step intervals (R = 1: the score pass hands over), S = 1, S
  larger than the ring would allow without deferral, a warm-up; matrices on
  the vector and the element path;
* the same runs equal the eager runner (the packed buffer accumulated every
  step, bf16 first-step stage) bit for bit;
* degenerate selections (k = 0, k = m) on one-element, one-row and
  one-column matrices;
* the entry point's host-side checks.
"""
import sys

import numpy as np
import pytest
import torch

import oracle as O
from tests._gpu import bits_np, f32_np, mask_np, same_bits
from workloads import derive_seed, gradient, master_weights, space_boundary

pytestmark = pytest.mark.gpu

zf = pytest.importorskip("paper_2505_12242_amd")
CM = zf.CHANNEL_MAJOR
RM = zf.ROW_MAJOR
HP = zf.AdamHparams(lr=1e-3)
# channel-major: n % 8 != 0 (43 x 77, 16 x 3 has 16 rows but 3 channels)
# takes the element path; row-major: every width but none a multiple of 8
SHAPES = [(264, 300), (4104, 70), (43, 77), (40, 1500), (16, 3)]
# storage variant -> layout
VARIANTS = {"cm": CM, "rm-vec": RM, "rm-col": RM}


def store(G, variant):
    """A logical [n, m] tensor in the variant's storage: channel-major
    transposed; rm-vec with rows padded to 16 bytes; rm-col contiguous."""
    if variant == "cm":
        return G.t().contiguous()
    if variant == "rm-vec":
        n, m = G.shape
        return zf.alloc_stored(RM, n, m, G.dtype, G.device).copy_(G)
    return G.contiguous()


def inputs(shapes, nslots, seed, ratio=0.1, variant="cm"):
    dev = torch.device("cuda")
    slots, host = [], []
    for s in range(nslots):
        buf, hb = [], []
        for q, (n, m) in enumerate(shapes):
            g = torch.Generator().manual_seed(derive_seed(seed, q, "scales"))
            sc = torch.exp(1.5 * torch.randn(m, generator=g, dtype=torch.float64))
            sc = space_boundary(sc * (1.0 + 0.01 * s), O.k_from_ratio(ratio, m))
            G = gradient(n, m, sc, derive_seed(seed, q, "g", s), device=dev)
            hb.append(bits_np(G))
            buf.append(store(G, variant))
        slots.append(buf)
        host.append(hb)
    weights, w0 = [], []
    for q, (n, m) in enumerate(shapes):
        w = master_weights(n, m, derive_seed(seed, q, "w"), device=dev).to(torch.bfloat16)
        w0.append(bits_np(w))
        weights.append(w.t().contiguous() if variant == "cm" else w.contiguous())
    return slots, host, weights, w0


def logical_of(variant):
    if variant == "cm":
        return lambda t: t.t().contiguous()
    return lambda t: t.contiguous()


SCHEDULES = [(4, 4, 0), (6, 4, 0), (1, 4, 0), (8, 3, 0), (2, 1, 0), (16, 6, 0), (4, 4, 2)]


@pytest.mark.timeout(600)
@pytest.mark.parametrize("variant", list(VARIANTS))
@pytest.mark.parametrize("R,S,warmup", SCHEDULES, ids=[f"R{r}S{s}w{w}" for r, s, w in SCHEDULES])
def test_deferred_runner_equals_oracle_and_eager(R, S, warmup, variant):
    T = 14
    nslots = max(3, min(S, R))
    slots, host, weights, w0 = inputs(SHAPES, nslots, derive_seed("deferred", R, S),
                                      variant=variant)
    logical = logical_of(variant)
    dev = torch.device("cuda")
    runs = {}
    for mode in ("deferred", "eager"):
        ws = [w.clone() for w in weights]
        runner = zf.SelectiveUpdateRunner(SHAPES, 0.1, HP, R, S, slots, ws, device=dev,
                                          layout=VARIANTS[variant], warmup=warmup,
                                          deferred_pack=(mode == "deferred"))
        assert runner.deferred == (mode == "deferred")
        orcs = [O.MatrixOracle(O.widen(w0[q]), w0[q], 0.1, HP.lr, HP.beta1, HP.beta2, HP.eps,
                               HP.weight_decay, R, S, warmup) for q in range(len(SHAPES))]
        out = []
        for t in range(1, T + 1):
            kind = runner.step()
            torch.cuda.synchronize()
            print(f"# deferred {variant} R={R} S={S} {mode} step {t} {kind}", file=sys.stderr,
                  flush=True)
            slot = (t - 1) % nslots
            for q in range(len(SHAPES)):
                ref = orcs[q].step(host[slot][q])
                assert ref["kind"] == O.schedule(t, R, S, warmup)
                assert (kind.refresh, kind.step_in_interval, kind.interval_end) == \
                    (ref["kind"].refresh, ref["kind"].step_in_interval, ref["kind"].interval_end)
                sel = runner.selection[q]
                assert np.array_equal(sel.sel_idx.cpu().numpy(), orcs[q].sel.sel), (q, t)
                assert np.array_equal(mask_np(sel.mask), orcs[q].sel.mask), (q, t)
                P, M, V = (f32_np(logical(x)) for x in runner.state[q])
                assert same_bits(P, orcs[q].P) and same_bits(M, orcs[q].M) and \
                    same_bits(V, orcs[q].V), (mode, q, t)
                W = bits_np(logical(ws[q]))
                assert np.array_equal(W, orcs[q].W), (mode, q, t)
                out.append(W)
                out.extend([P, M, V])
                if kind.interval_end:
                    D = f32_np(logical(runner.unpacked[q]))
                    assert same_bits(D, ref["unpacked"]), (mode, q, t)
                    out.append(D)
        runner.close()
        runs[mode] = out
    assert len(runs["deferred"]) == len(runs["eager"])
    for a, b in zip(runs["deferred"], runs["eager"]):
        assert same_bits(a, b)


# one element, one row, one column, a whole mask word, a square of 8, and
# 3 channels of 16 rows (channel-major element path)
EDGE_SHAPES = [(1, 1), (1, 9), (5, 1), (9, 64), (8, 8), (16, 3)]


@pytest.mark.timeout(300)
@pytest.mark.parametrize("variant", list(VARIANTS))
@pytest.mark.parametrize("ratio", [0.0, 1.0, 0.5])
def test_deferred_degenerate_selections(ratio, variant):
    """k = 0 (the hand-over is the whole interval's sum, no Adam), k = m
    (the hand-over is all +0.0 and no gradient is summed) and k = m / 2, on
    one-element, one-row and one-column matrices, over R = 6, S = 4 (an
    interval cut short by a refresh): the deferred runner equals the oracle
    and the eager runner bit for bit at every step."""
    R, S, T = 6, 4, 9
    nslots = 4
    slots, host, weights, w0 = inputs(EDGE_SHAPES, nslots, derive_seed("deferred-edge", ratio),
                                      ratio=ratio, variant=variant)
    logical = logical_of(variant)
    dev = torch.device("cuda")
    runs = {}
    for mode in ("deferred", "eager"):
        ws = [w.clone() for w in weights]
        runner = zf.SelectiveUpdateRunner(EDGE_SHAPES, ratio, HP, R, S, slots, ws, device=dev,
                                          layout=VARIANTS[variant],
                                          deferred_pack=(mode == "deferred"))
        orcs = [O.MatrixOracle(O.widen(w0[q]), w0[q], ratio, HP.lr, HP.beta1, HP.beta2, HP.eps,
                               HP.weight_decay, R, S) for q in range(len(EDGE_SHAPES))]
        out = []
        for t in range(1, T + 1):
            kind = runner.step()
            torch.cuda.synchronize()
            print(f"# deferred edges {variant} ratio={ratio} {mode} step {t} {kind}",
                  file=sys.stderr, flush=True)
            slot = (t - 1) % nslots
            for q in range(len(EDGE_SHAPES)):
                ref = orcs[q].step(host[slot][q])
                sel = runner.selection[q]
                assert np.array_equal(sel.sel_idx.cpu().numpy(), orcs[q].sel.sel), (q, t)
                P, M, V = (f32_np(logical(x)) for x in runner.state[q])
                assert same_bits(P, orcs[q].P) and same_bits(M, orcs[q].M) and \
                    same_bits(V, orcs[q].V), (mode, q, t)
                W = bits_np(logical(ws[q]))
                assert np.array_equal(W, orcs[q].W), (mode, q, t)
                out.extend([W, P, M, V])
                if kind.interval_end:
                    D = f32_np(logical(runner.unpacked[q]))
                    assert same_bits(D, ref["unpacked"]), (mode, q, t)
                    if ratio == 1.0:
                        assert not np.any(D.view(np.uint32)), (mode, q, t)  # all +0.0
                    out.append(D)
        runner.close()
        runs[mode] = out
    for a, b in zip(runs["deferred"], runs["eager"]):
        assert same_bits(a, b)


def test_deferred_needs_the_interval_in_the_ring():
    slots, _, weights, _ = inputs(SHAPES[:2], 3, 5)
    with pytest.raises(ValueError, match="gradient slots"):
        zf.SelectiveUpdateRunner(SHAPES[:2], 0.1, HP, 4, 4, slots, weights, layout=CM,
                                 deferred_pack=True)
    # Zen-auto with deferred packing: decided on the device, channel-major only
    with pytest.raises(ValueError, match="fixed schedule"):
        zf.SelectiveUpdateRunner(SHAPES[:2], 0.1, HP, 4, 4, slots, weights, layout=CM,
                                 zen_tau=1.0, zen_on_device=False, deferred_pack=True)
    rslots, _, rweights, _ = inputs(SHAPES[:2], 4, 5, variant="rm-col")
    with pytest.raises(ValueError, match="fixed schedule"):
        zf.SelectiveUpdateRunner(SHAPES[:2], 0.1, HP, 4, 4, rslots, rweights, layout=RM,
                                 zen_tau=1.0, deferred_pack=True)


@pytest.mark.parametrize("variant", list(VARIANTS))
def test_deferred_entry_point_checks(variant):
    """Host-side checks of zf_plan_update_handover_deferred: the earlier
    plans must cover the same matrices (count, shapes, k; channel-major:
    access path), at most 15 of them; nothing is enqueued otherwise."""
    dev = torch.device("cuda")
    lay = VARIANTS[variant]
    slots, _, weights, _ = inputs(SHAPES[:2], 4, 6, variant=variant)
    runner = zf.SelectiveUpdateRunner(SHAPES[:2], 0.1, HP, 4, 4, slots, weights, device=dev,
                                      layout=lay, deferred_pack=True)
    runner.step()
    plan = runner.plans[1][runner.cur][0]
    earlier = [runner.plans[0][runner.cur][0]]
    before = [x.clone() for x in runner.unpacked]
    other = zf.SelectiveUpdateRunner(SHAPES[:1], 0.1, HP, 4, 4, [s[:1] for s in slots],
                                     [w.clone() for w in weights[:1]], device=dev, layout=lay,
                                     deferred_pack=True)
    for bad in ([other.plans[0][0][0]],            # another matrix count
                earlier * 16):                      # more than 15 earlier steps
        with pytest.raises(zf.ZfError, match="invalid argument"):
            plan.update_handover_deferred(HP, 2, bad, 0.5)
    with pytest.raises(zf.ZfError, match="invalid argument"):
        plan.update_handover_deferred(HP, 2, earlier, float("nan"))
    torch.cuda.synchronize()
    for a, b in zip(before, runner.unpacked):
        assert torch.equal(a.view(torch.int32), b.view(torch.int32))
    other.close()
    runner.close()
