"""Plain CPU oracle of the selective-update hot path (TEST INFRASTRUCTURE).

Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may
import this module.  The product path never calls it, and it shares no code
with the HIP library or its Python binding.

It restates, in slow and direct numpy, what ZenFlow's GPU side computes for
one weight matrix (paper: "ZenFlow Design", Asynchronous Offloading Workflow
and Gradient Selection; Convergence Analysis for the accumulate-then-apply
rule):

* colnorm     -- per-input-channel squared gradient norm (Gradient Selection,
                 "Lightweight Proxy for Gradient Ranking").  The definition,
                 summed in fp64 in row order and rounded once to fp32.
* select_topk -- the k columns with the largest score (Problem #3 top-k
                 selection applied to channels).  A plain sort.
* remap       -- states follow their columns when the selection is refreshed
                 (selective optimizer initialised only with the chosen
                 subset; swap-in of states, Zero-stall Pipeline).
* adam_selected -- Adam (Kingma & Ba) / AdamW decoupled decay on the selected
                 columns' fp32 master, first and second moments, in place,
                 then the bf16 write-back (Asynchronous Offloading Workflow,
                 Implementation "Selective GPU-side Optimizer").
* pack_accumulate / unpack -- unselected columns summed over an interval of
                 S steps and handed over as one dense buffer (Asynchronous
                 Offloading Workflow; the S-step rule of the Convergence
                 Analysis, whose 1/S mean is unpack's scale).
* schedule    -- which step refreshes the selection, starts or ends an
                 accumulation interval.
* swap_states / deferred_adam / OffloadOracle -- the offloaded optimizer:
                 a full-state store backs the selective optimizer (states of
                 columns leaving the selection are swapped out to it, those
                 of entering columns swapped in, Zero-stall Pipeline
                 "Swapping out/in"), and at every interval end the
                 accumulated mean gradient updates the unselected columns
                 from the store (Asynchronous Offloading Workflow; the
                 delayed-coordinate rule of the Convergence Analysis).
* Zen-auto    -- the adaptive interval (Zero-stall Pipeline, "Hyperparameter
                 Auto-tuning"): channel norms of the accumulated buffer and of
                 the selected channels' gradient, their means over the whole
                 gradient set, and a trigger that ends the interval early
                 (column_sq_norms, zen_auto_stats, zen_auto_trigger,
                 ZenAutoOracle).

Precision.  The workloads fix fp32 master weights, moments and accumulation
buffer, and the selective optimizer extends PyTorch's fp32 Adam
(Implementation).  So Adam, pack and unpack are written as IEEE fp32
operations, one rounding per operation, in the order given in each function
(numpy float32 ufuncs: no fused multiply-add, correctly rounded sqrt and
division, subnormals kept).  Column norms are summed in fp64.  Every
function is pinned by tests/test_oracle_*.py against closed forms, brute
force, exact rational arithmetic, library routines or invariants.
"""

from __future__ import annotations

import math
from dataclasses import dataclass
from typing import Optional, Tuple

import numpy as np

__all__ = [
    "Selection", "AdamConsts", "StepKind",
    "widen", "bf16_round", "colnorm", "k_from_ratio", "select_topk",
    "slots_of", "remap", "adam_selected", "pack_accumulate", "unpack",
    "schedule", "MatrixOracle",
    "column_sq_norms", "zen_auto_stats", "ZenAutoTotals", "zen_auto_trigger",
    "ZenAutoOracle",
    "swap_states", "deferred_adam", "OffloadOracle",
]


# ---------------------------------------------------------------------------
# bf16 <-> fp32 (BF16 training: parameters and gradients in bf16, Background
# "Training Memory Breakdown")
# ---------------------------------------------------------------------------

def widen(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) -> fp32: the bf16 bits are the top half of
    an fp32 word, so the widening is exact."""
    b = np.asarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def bf16_round(x: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bit patterns, round to nearest, ties to even.  NaN stays
    NaN (quiet bit set); overflow past the largest bf16 gives infinity."""
    u = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    is_nan = (u & 0x7FFFFFFF) > 0x7F800000
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16) & 0xFFFF
    r = np.where(is_nan, ((u >> 16) | 0x40) & 0xFFFF, r)
    return r.astype(np.uint16)


# ---------------------------------------------------------------------------
# a1: column scores
# ---------------------------------------------------------------------------

def colnorm(G: np.ndarray) -> np.ndarray:
    """s_j = sum_i g_ij^2 over the rows of an n x m bf16 gradient (uint16
    bits), one score per input channel j (Gradient Selection, "Lightweight
    Proxy": per-column squared norms).  Squares of bf16 values are exact in
    fp64; the fp64 row-order sum is rounded once to fp32."""
    G = np.asarray(G, dtype=np.uint16)
    n, m = G.shape
    acc = np.zeros(m, dtype=np.float64)
    for i in range(n):
        g = widen(G[i]).astype(np.float64)
        acc += g * g
    return acc.astype(np.float32)


# ---------------------------------------------------------------------------
# a2: top-k selection
# ---------------------------------------------------------------------------

def k_from_ratio(ratio: float, m: int) -> int:
    """Number of selected columns for a top-k ratio (Evaluation, ZenFlow
    hyperparameters "topk_ratio").  Reading: round half up, k = floor(ratio*m
    + 1/2) in double, clamped to [0, m]."""
    if not (0.0 <= ratio <= 1.0) or m < 0:
        raise ValueError("ratio must lie in [0, 1] and m >= 0")
    return max(0, min(m, int(math.floor(ratio * m + 0.5))))


@dataclass
class Selection:
    sel: np.ndarray      # int32 [k], ascending column indices
    unsel: np.ndarray    # int32 [m-k], ascending column indices
    mask: np.ndarray     # uint64 [ceil(m/64)], bit b of word w <=> column 64w+b selected
    prefix: np.ndarray   # int32 [ceil(m/64)], selected columns with index < 64w
    m: int

    @property
    def k(self) -> int:
        return int(self.sel.size)


def _mask_and_prefix(sel: np.ndarray, m: int) -> Tuple[np.ndarray, np.ndarray]:
    words = (m + 63) // 64
    mask = np.zeros(words, dtype=np.uint64)
    for j in sel.tolist():
        mask[j // 64] |= np.uint64(1) << np.uint64(j % 64)
    prefix = np.zeros(words, dtype=np.int32)
    count = 0
    for w in range(words):
        prefix[w] = count
        count += bin(int(mask[w])).count("1")
    return mask, prefix


def select_topk(scores: np.ndarray, k: int) -> Selection:
    """The k columns with the largest score.  Order: larger score first, and
    among equal scores (-0.0 equals +0.0) the lower column index first; the
    chosen set and its complement are returned in ascending index order."""
    s = np.asarray(scores, dtype=np.float32)
    m = int(s.size)
    if not 0 <= k <= m:
        raise ValueError("k must lie in [0, m]")
    idx = np.arange(m)
    # np.lexsort sorts by the last key first: descending score, then index.
    order = np.lexsort((idx, -s.astype(np.float64)))
    sel = np.sort(order[:k]).astype(np.int32)
    unsel = np.sort(order[k:]).astype(np.int32)
    mask, prefix = _mask_and_prefix(sel, m)
    return Selection(sel, unsel, mask, prefix, m)


def slots_of(cols: np.ndarray, m: int) -> np.ndarray:
    """slot[j] = position of column j in the ascending list `cols`, -1 if
    absent (row-compact layout: slot r of a row <-> column cols[r])."""
    slot = np.full(m, -1, dtype=np.int64)
    slot[np.asarray(cols, dtype=np.int64)] = np.arange(len(cols))
    return slot


# ---------------------------------------------------------------------------
# a3 + a4: Adam on the selected columns and bf16 write-back
# ---------------------------------------------------------------------------

@dataclass(frozen=True)
class AdamConsts:
    """Per-step constants, each computed in double and rounded once to fp32."""
    B1: np.float32
    B2: np.float32
    C1: np.float32
    C2: np.float32
    LR: np.float32
    EPS: np.float32
    WD: np.float32     # lr * weight_decay (AdamW decoupled decay)
    IB1: np.float32    # 1 / (1 - beta1^t)
    IB2: np.float32    # 1 / (1 - beta2^t)

    @staticmethod
    def at_step(lr: float, beta1: float, beta2: float, eps: float,
                weight_decay: float, t: int) -> "AdamConsts":
        if t < 1:
            raise ValueError("the step counter is 1-based")
        f = np.float32
        return AdamConsts(
            B1=f(beta1), B2=f(beta2), C1=f(1.0 - beta1), C2=f(1.0 - beta2),
            LR=f(lr), EPS=f(eps), WD=f(lr * weight_decay),
            IB1=f(1.0 / (1.0 - beta1 ** t)), IB2=f(1.0 / (1.0 - beta2 ** t)))


def adam_selected(G: np.ndarray, sel: np.ndarray, P: np.ndarray, M: np.ndarray,
                  V: np.ndarray, c: AdamConsts):
    """One Adam/AdamW step on the selected columns.

    G: bf16 gradient bits [n, m]; sel: ascending selected columns [k];
    P, M, V: row-compact fp32 states [n, k] (slot r <-> column sel[r]).
    Returns (P', M', V', W_sel) with W_sel the bf16 bits of P' for the
    selected columns.  Each line is one fp32 operation per element:

        m' = B1*m + C1*g
        v' = B2*v + C2*(g*g)
        d  = sqrt(v'*IB2) + EPS            (IB2 = 1/(1-beta2^t))
        u  = (m'*IB1) / d                  (IB1 = 1/(1-beta1^t))
        p  = p - WD*p                      (only when weight decay != 0)
        p' = p - LR*u
        w  = bf16(p')
    """
    g = widen(np.asarray(G)[:, np.asarray(sel, dtype=np.int64)])
    P = np.asarray(P, dtype=np.float32)
    M = np.asarray(M, dtype=np.float32)
    V = np.asarray(V, dtype=np.float32)
    m1 = c.B1 * M + c.C1 * g
    v1 = c.B2 * V + c.C2 * (g * g)
    d = np.sqrt(v1 * c.IB2) + c.EPS
    u = (m1 * c.IB1) / d
    p = P - c.WD * P if c.WD != 0 else P
    p1 = p - c.LR * u
    return p1.astype(np.float32), m1.astype(np.float32), v1.astype(np.float32), bf16_round(p1)


def remap(prev: Optional[Selection], new: Selection, P: Optional[np.ndarray],
          M: Optional[np.ndarray], V: Optional[np.ndarray], W: np.ndarray,
          master: Optional[np.ndarray] = None):
    """Compact states for a new selection.  A column that stays selected keeps
    its (p, m, v) -- moved to its new slot; a newly selected column starts
    with m = v = 0 and p taken from the fp32 `master` [n, m] when given, else
    from the widened bf16 weight W [n, m].  `prev` None means no column was
    selected before."""
    W = np.asarray(W, dtype=np.uint16)
    n = W.shape[0]
    k = new.k
    P2 = np.zeros((n, k), dtype=np.float32)
    M2 = np.zeros((n, k), dtype=np.float32)
    V2 = np.zeros((n, k), dtype=np.float32)
    old_slot = slots_of(prev.sel, new.m) if prev is not None else np.full(new.m, -1)
    for r, j in enumerate(new.sel.tolist()):
        ro = int(old_slot[j])
        if ro >= 0:
            P2[:, r] = P[:, ro]
            M2[:, r] = M[:, ro]
            V2[:, r] = V[:, ro]
        elif master is not None:
            P2[:, r] = np.asarray(master, dtype=np.float32)[:, j]
        else:
            P2[:, r] = widen(W[:, j])
    return P2, M2, V2


# ---------------------------------------------------------------------------
# a5 + a6: accumulation of the unselected columns, hand-over
# ---------------------------------------------------------------------------

def pack_accumulate(G: np.ndarray, unsel: np.ndarray, A: Optional[np.ndarray],
                    step_in_interval: int) -> np.ndarray:
    """A[i, u] = g[i, unsel[u]] on the first step of an interval, else
    A[i, u] + g[i, unsel[u]] (one fp32 addition).  Row-compact [n, m-k]."""
    g = widen(np.asarray(G)[:, np.asarray(unsel, dtype=np.int64)])
    if step_in_interval < 1:
        raise ValueError("step_in_interval is 1-based")
    if step_in_interval == 1:
        return g.copy()
    return (np.asarray(A, dtype=np.float32) + g).astype(np.float32)


def unpack(A: np.ndarray, sel: Selection, scale: float = 1.0) -> np.ndarray:
    """Dense [n, m] fp32: +0.0 at selected columns, scale * A[i, u] at the
    unselected column unsel[u] (one fp32 multiply; scale 1 copies)."""
    A = np.asarray(A, dtype=np.float32)
    n = A.shape[0]
    D = np.zeros((n, sel.m), dtype=np.float32)
    D[:, sel.unsel.astype(np.int64)] = A * np.float32(scale)
    return D


# ---------------------------------------------------------------------------
# schedule
# ---------------------------------------------------------------------------

@dataclass(frozen=True)
class StepKind:
    refresh: bool           # recompute scores and the selection at this step
    step_in_interval: int   # 1 = first step of an accumulation interval
    interval_end: bool      # hand the accumulated buffer over after this step


def _is_refresh(t: int, R: int) -> bool:
    return (t - 1) % R == 0


def _is_start(t: int, R: int, S: int, warmup: int = 0) -> bool:
    if t <= warmup + 1:
        return True
    return _is_refresh(t, R) or (t - warmup - 1) % S == 0


def schedule(t: int, R: int, S: int, warmup: int = 0) -> StepKind:
    """Step kinds for 1-based step t, selection refresh interval R and
    accumulation interval S.  Reading: the selection is recomputed when
    (t-1) mod R = 0 (index reuse between refreshes, Gradient Selection
    "Temporal Locality"); an interval starts every S steps (the t mod S rule
    of the Convergence Analysis) and also at every refresh, because the packed
    layout follows the selection; an interval ends right before the next
    one starts.

    warmup = tau: the first tau steps are synchronous (Convergence Analysis,
    "Warm-up mitigates early-stage staleness"), read as intervals of one
    step -- the unselected part is handed over after every step, so it is
    never stale -- and the S-step intervals count from step tau + 1."""
    if t < 1 or R < 1 or S < 1 or warmup < 0:
        raise ValueError("t, R and S are 1-based / positive, warmup >= 0")
    start = t
    while not _is_start(start, R, S, warmup):
        start -= 1
    return StepKind(refresh=_is_refresh(t, R), step_in_interval=t - start + 1,
                    interval_end=_is_start(t + 1, R, S, warmup))


# ---------------------------------------------------------------------------
# one matrix across steps
# ---------------------------------------------------------------------------

class MatrixOracle:
    """Runs the per-step composition for one weight matrix:
    refresh -> colnorm, select_topk, remap; every step -> adam_selected and
    pack_accumulate; interval end -> unpack with scale 1/(interval length)
    (the 1/S mean of the Convergence Analysis)."""

    def __init__(self, master: np.ndarray, W: np.ndarray, ratio: float,
                 lr: float, beta1: float, beta2: float, eps: float,
                 weight_decay: float, R: int, S: int, warmup: int = 0):
        self.warmup = warmup
        self.master = np.asarray(master, dtype=np.float32)
        self.W = np.array(W, dtype=np.uint16, copy=True)
        self.n, self.m = self.W.shape
        self.k = k_from_ratio(ratio, self.m)
        self.hyper = (lr, beta1, beta2, eps, weight_decay)
        self.R, self.S = R, S
        self.t = 0
        self.sel: Optional[Selection] = None
        self.P = self.M = self.V = None
        self.A: Optional[np.ndarray] = None

    def step(self, G: np.ndarray) -> dict:
        """One step of the fixed schedule (refresh every R steps, intervals
        of S steps after `warmup` one-step intervals)."""
        kind = schedule(self.t + 1, self.R, self.S, self.warmup)
        out = self.advance(G, kind.refresh, kind.step_in_interval)
        out["kind"] = kind
        if kind.interval_end:
            out["unpacked"] = self.hand_over(kind.step_in_interval)
        return out

    def advance(self, G: np.ndarray, refresh: bool, step_in_interval: int) -> dict:
        """Everything of a step up to the hand-over: scores, selection and
        state remap when `refresh`, then Adam on the selected columns and the
        accumulation of the others (`step_in_interval` = 1 overwrites)."""
        self.t += 1
        out = {}
        if refresh:
            s = colnorm(G)
            new = select_topk(s, self.k)
            first = self.sel is None
            self.P, self.M, self.V = remap(self.sel, new, self.P, self.M, self.V,
                                           self.W, self.master if first else None)
            self.sel = new
            out["norms"] = s
        elif self.sel is None:
            raise ValueError("the first step must refresh the selection")
        c = AdamConsts.at_step(*self.hyper, self.t)
        self.P, self.M, self.V, wsel = adam_selected(G, self.sel.sel, self.P, self.M,
                                                     self.V, c)
        self.W[:, self.sel.sel.astype(np.int64)] = wsel
        self.A = pack_accumulate(G, self.sel.unsel, self.A, step_in_interval)
        return out

    def hand_over(self, steps: int) -> np.ndarray:
        """The dense hand-over buffer of an interval of `steps` steps, scaled
        by the fp32 value of 1/steps (the mean of the Convergence Analysis)."""
        return unpack(self.A, self.sel, float(np.float32(1.0 / steps)))


# ---------------------------------------------------------------------------
# Offloaded optimizer states: swap at a refresh, deferred host update
# ---------------------------------------------------------------------------

def swap_states(prev: Optional[Selection], new: Selection, P: Optional[np.ndarray],
                M: Optional[np.ndarray], V: Optional[np.ndarray], store):
    """Compact states for a new selection when a full-state store (the
    offloaded optimizer's fp32 master, first and second moments of every
    column, [n, m] each) backs the selective optimizer (Zero-stall Pipeline,
    "Swapping out/in"):

    * a column selected before and after keeps its compact (p, m, v), moved
      to its new slot;
    * a column that leaves the selection writes its compact (p, m, v) back to
      its column of the store (swap-out);
    * a column that enters reads (p, m, v) from its column of the store
      (swap-in).

    Leaving and entering columns are disjoint, so the order of the two
    copies does not matter.  `prev` None means nothing was selected before.
    Returns (P2, M2, V2, store2) with store2 a new (SP, SM, SV) tuple."""
    SP, SM, SV = (np.array(x, dtype=np.float32, copy=True) for x in store)
    n = SP.shape[0]
    old_slot = slots_of(prev.sel, new.m) if prev is not None else np.full(new.m, -1)
    new_slot = slots_of(new.sel, new.m)
    if prev is not None:
        for ro, j in enumerate(prev.sel.tolist()):
            if new_slot[j] < 0:
                SP[:, j] = P[:, ro]
                SM[:, j] = M[:, ro]
                SV[:, j] = V[:, ro]
    k = new.k
    P2 = np.zeros((n, k), dtype=np.float32)
    M2 = np.zeros((n, k), dtype=np.float32)
    V2 = np.zeros((n, k), dtype=np.float32)
    for r, j in enumerate(new.sel.tolist()):
        ro = int(old_slot[j])
        if ro >= 0:
            P2[:, r], M2[:, r], V2[:, r] = P[:, ro], M[:, ro], V[:, ro]
        else:
            P2[:, r], M2[:, r], V2[:, r] = SP[:, j], SM[:, j], SV[:, j]
    return P2, M2, V2, (SP, SM, SV)


def deferred_adam(A: np.ndarray, unsel: np.ndarray, scale: float, store, c: AdamConsts):
    """The deferred update of the unselected columns (Asynchronous Offloading
    Workflow: the accumulated unimportant gradients are applied by the
    offloaded optimizer; Convergence Analysis: the delayed coordinates move
    by the mean of the S accumulated gradients).  For every unselected
    column j = unsel[u] and every row i:

        g = A[i, u] * scale        (one fp32 multiply; scale = fp32(1/S)
                                    gives the interval's mean gradient)

    followed by the Adam/AdamW sequence of adam_selected on the store's
    (p, m, v) of column j, with the constants `c` of the offloaded
    optimizer's own step.  Returns (store2, W_unsel) with W_unsel the bf16
    bits [n, m-k] of the new master of the unselected columns (slot order);
    selected columns of the store are unchanged."""
    SP, SM, SV = (np.array(x, dtype=np.float32, copy=True) for x in store)
    cols = np.asarray(unsel, dtype=np.int64)
    g = np.asarray(A, dtype=np.float32) * np.float32(scale)
    p0, m0, v0 = SP[:, cols], SM[:, cols], SV[:, cols]
    m1 = c.B1 * m0 + c.C1 * g
    v1 = c.B2 * v0 + c.C2 * (g * g)
    d = np.sqrt(v1 * c.IB2) + c.EPS
    u = (m1 * c.IB1) / d
    p = p0 - c.WD * p0 if c.WD != 0 else p0
    p1 = (p - c.LR * u).astype(np.float32)
    SP[:, cols], SM[:, cols], SV[:, cols] = p1, m1.astype(np.float32), v1.astype(np.float32)
    return (SP, SM, SV), bf16_round(p1)


class OffloadOracle:
    """One matrix under the whole method with offloaded optimizer states.
    The store holds every column's (p, m, v) -- initially the fp32 master
    and zero moments.  A refresh scores, selects and swaps states against
    the store (swap_states); every step updates the selected columns (the
    selective optimizer, global step t) and accumulates the others; every
    interval end applies the deferred update (deferred_adam with scale
    fp32(1/length), constants of the offloaded optimizer's own step counter
    th = 1, 2, ... -- one step per hand-over, reading) and writes the new
    bf16 weights of the unselected columns into W.  The hand-over is applied
    before the next step: an implementation that overlaps it with later
    steps must give the same result, which holds when it lands before the
    next refresh (only a refresh reads the store; only the unselected
    columns of W change)."""

    def __init__(self, master: np.ndarray, W: np.ndarray, ratio: float, lr: float,
                 beta1: float, beta2: float, eps: float, weight_decay: float, R: int, S: int,
                 warmup: int = 0):
        self.warmup = warmup
        master = np.asarray(master, dtype=np.float32)
        self.W = np.array(W, dtype=np.uint16, copy=True)
        self.n, self.m = self.W.shape
        self.k = k_from_ratio(ratio, self.m)
        self.hyper = (lr, beta1, beta2, eps, weight_decay)
        self.R, self.S = R, S
        self.t = 0
        self.th = 0
        self.sel: Optional[Selection] = None
        self.P = self.M = self.V = None
        self.A: Optional[np.ndarray] = None
        z = np.zeros_like(master)
        self.store = (master.copy(), z, z.copy())

    def step(self, G: np.ndarray) -> dict:
        """One step of the fixed schedule (refresh every R steps, intervals
        of S steps after `warmup` one-step intervals), the deferred update
        at every interval end."""
        kind = schedule(self.t + 1, self.R, self.S, self.warmup)
        out = self.advance(G, kind.refresh, kind.step_in_interval)
        out["kind"] = kind
        if kind.interval_end:
            out["weight_cols"] = self.hand_over(kind.step_in_interval)
        return out

    def advance(self, G: np.ndarray, refresh: bool, step_in_interval: int) -> dict:
        """Everything of a step before the hand-over: scores, selection and
        the swap against the store when `refresh`, then Adam on the selected
        columns and the accumulation of the others."""
        self.t += 1
        out = {}
        if refresh:
            s = colnorm(G)
            new = select_topk(s, self.k)
            self.P, self.M, self.V, self.store = swap_states(self.sel, new, self.P, self.M,
                                                             self.V, self.store)
            self.sel = new
            out["norms"] = s
        elif self.sel is None:
            raise ValueError("the first step must refresh the selection")
        c = AdamConsts.at_step(*self.hyper, self.t)
        self.P, self.M, self.V, wsel = adam_selected(G, self.sel.sel, self.P, self.M, self.V, c)
        self.W[:, self.sel.sel.astype(np.int64)] = wsel
        self.A = pack_accumulate(G, self.sel.unsel, self.A, step_in_interval)
        return out

    def hand_over(self, steps: int) -> np.ndarray:
        """The deferred update at the end of an interval of `steps` steps
        (scale fp32(1/steps), the offloaded optimizer's next step); returns
        the new bf16 weights of the unselected columns, also written into W."""
        self.th += 1
        ch = AdamConsts.at_step(*self.hyper, self.th)
        scale = float(np.float32(1.0 / steps))
        self.store, wun = deferred_adam(self.A, self.sel.unsel, scale, self.store, ch)
        self.W[:, self.sel.unsel.astype(np.int64)] = wun
        return wun


# ---------------------------------------------------------------------------
# Zen-auto: adaptive accumulation interval
# ---------------------------------------------------------------------------

def column_sq_norms(X: np.ndarray) -> np.ndarray:
    """Squared norm of every column of an fp32 matrix: squares of fp32 values
    are exact in fp64 (24-bit significands), the fp64 row-order sum is
    rounded once to fp32 (the same definition as colnorm, for fp32 data)."""
    X = np.asarray(X, dtype=np.float32)
    acc = np.zeros(X.shape[1], dtype=np.float64)
    for i in range(X.shape[0]):
        x = X[i].astype(np.float64)
        acc += x * x
    return acc.astype(np.float32)


def zen_auto_stats(G: np.ndarray, sel: Selection, A: np.ndarray) -> Tuple[np.ndarray, np.ndarray]:
    """Per-channel quantities Zen-auto tracks (Zero-stall Pipeline,
    "Hyperparameter Auto-tuning"), taken after a step's accumulation:
    sel_sq[r] = squared norm of this step's gradient column sel[r] (the
    important part), acc_sq[u] = squared norm of the accumulated column in
    packed slot u (the unimportant part).  Reading: the important part is
    measured on the current step's gradient, which the selective optimizer
    applies at once."""
    g = widen(np.asarray(G)[:, np.asarray(sel.sel, dtype=np.int64)])
    return column_sq_norms(g), column_sq_norms(A)


@dataclass(frozen=True)
class ZenAutoTotals:
    sum_sel: float   # sum over every selected channel of its norm
    k: int           # selected channels
    sum_acc: float   # sum over every unselected channel of its accumulated norm
    u: int           # unselected channels
    trigger: bool


def zen_auto_trigger(stats, tau: float) -> ZenAutoTotals:
    """Zen-auto's decision over a whole gradient set (a list of
    (sel_sq, acc_sq) per matrix).  The mean accumulated channel norm of the
    unimportant part, sum_acc / u, is compared with the mean channel norm of
    the important part, sum_sel / k.  Reading of "comparable": the hand-over
    is triggered when sum_acc / u >= tau * sum_sel / k, evaluated without
    division as sum_acc * k >= (tau * sum_sel) * u in fp64; norms are the fp64
    square roots of the fp32 squared norms, summed in fp64 matrix by matrix
    in slot order.  No trigger when either part is empty."""
    sum_sel = 0.0
    sum_acc = 0.0
    k = u = 0
    for sel_sq, acc_sq in stats:
        for x in np.asarray(sel_sq, dtype=np.float32):
            sum_sel += math.sqrt(float(x))
        for x in np.asarray(acc_sq, dtype=np.float32):
            sum_acc += math.sqrt(float(x))
        k += len(sel_sq)
        u += len(acc_sq)
    trig = k > 0 and u > 0 and sum_acc * float(k) >= (float(tau) * sum_sel) * float(u)
    return ZenAutoTotals(sum_sel, k, sum_acc, u, bool(trig))


class ZenAutoOracle:
    """Several matrices under Zen-auto's adaptive interval (MatrixOracle:
    the hand-over is the dense buffer; OffloadOracle: the hand-over is the
    deferred update of the offloaded optimizer).  Reading of the
    schedule: the selection is refreshed when (t-1) mod R = 0 as in the fixed
    schedule; an interval starts at a refresh or after a hand-over, and ends
    (hand-over with scale 1/length) when the trigger fires, when it reaches
    S_max steps, or before a refresh.  Interval lengths count from the
    interval's start, not from a global t mod S grid; so with tau = +inf this
    is the fixed schedule with S = S_max whenever R is a multiple of S_max
    (or R = 1)."""

    def __init__(self, oracles, R: int, S_max: int, tau: float, warmup: int = 0):
        self.orcs = list(oracles)
        self.R, self.S_max, self.tau = R, S_max, tau
        self.warmup = warmup  # the first `warmup` steps hand over after every step
        self.t = 0
        self.length = 0
        self.ended = True

    def step(self, grads) -> dict:
        self.t += 1
        refresh = _is_refresh(self.t, self.R)
        self.length = 1 if (refresh or self.ended or self.t <= self.warmup) else self.length + 1
        outs = [o.advance(G, refresh, self.length) for o, G in zip(self.orcs, grads)]
        stats = [zen_auto_stats(G, o.sel, o.A) for o, G in zip(self.orcs, grads)]
        tot = zen_auto_trigger(stats, self.tau)
        end = (tot.trigger or self.length >= self.S_max or _is_refresh(self.t + 1, self.R)
               or self.t <= self.warmup)
        self.ended = end
        res = {"refresh": refresh, "step_in_interval": self.length, "interval_end": end,
               "totals": tot, "stats": stats, "outs": outs}
        if end:
            res["unpacked"] = [o.hand_over(self.length) for o in self.orcs]
        return res
