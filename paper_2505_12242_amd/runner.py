"""Per-step driver of the hot path over a set of weight matrices.

Owns the device buffers of every matrix (bf16 weight, compact fp32 states,
packed accumulation buffer, scores, selections, dense hand-over buffer) and
issues one batched launch per kernel per step:

    refresh step : zf_plan_colnorm -> zf_plan_topk_select ->
                   zf_plan_update (states remapped to the new selection)
    other steps  : zf_plan_update (states in place)
    interval end : zf_plan_unpack with scale 1/(steps in the interval)

Compact states and selections are double-buffered: a refresh writes the new
selection and new states into the other buffer while reading the previous
ones (ZF_STATES_REMAP), so a column that stays selected carries its moments
(the selective optimizer follows its subset, Zero-stall Pipeline "Swapping
out/in") without a separate pass.  Gradients come from caller-owned slots;
step t reads slot (t-1) mod len(slots).  Every tensor of the runner is
stored in one layout (ROW_MAJOR or CHANNEL_MAJOR, see the binding).
"""

from __future__ import annotations

from dataclasses import dataclass
from typing import List, Optional, Sequence, Tuple

import torch

from ._lib import (ROW_MAJOR, STATES_INIT, STATES_INPLACE, STATES_REMAP, AdamHparams,
                   MatrixBuffers, Plan, Selection, StateSource, _stored, k_from_ratio)


@dataclass(frozen=True)
class StepKind:
    refresh: bool
    step_in_interval: int
    interval_end: bool


def schedule(t: int, R: int, S: int) -> StepKind:
    """Refresh when (t-1) mod R == 0; an accumulation interval starts every S
    steps and at every refresh, and ends right before the next start."""
    if t < 1 or R < 1 or S < 1:
        raise ValueError("t, R and S must be >= 1")
    last_refresh = t - (t - 1) % R
    last_s_start = t - (t - 1) % S
    start = max(last_refresh, last_s_start)
    nxt = t + 1
    return StepKind(refresh=(t - 1) % R == 0, step_in_interval=t - start + 1,
                    interval_end=(nxt - 1) % R == 0 or (nxt - 1) % S == 0)


class _NoRecord:
    def __enter__(self):
        return self

    def __exit__(self, *exc):
        return False


def _no_record(name):
    return _NoRecord()


class SelectiveUpdateRunner:
    def __init__(self, shapes: Sequence[Tuple[int, int]], ratio: float, hp: AdamHparams,
                 refresh: int, accum: int, grad_slots: Sequence[Sequence[torch.Tensor]],
                 weights: Sequence[torch.Tensor],
                 init_master: Optional[Sequence[torch.Tensor]] = None,
                 device=None, keep_unpacked: bool = True, layout: int = ROW_MAJOR):
        self.device = torch.device(device) if device is not None else torch.device("cuda")
        self.shapes = [(int(n), int(m)) for n, m in shapes]
        self.ratio, self.hp, self.R, self.S = ratio, hp, int(refresh), int(accum)
        self.ks = [k_from_ratio(ratio, m) for _, m in self.shapes]
        self.layout = layout
        self.keep_unpacked = keep_unpacked
        self.weights = list(weights)
        self.init_master = list(init_master) if init_master is not None else None
        dev = self.device
        f32 = torch.float32
        self.sels: List[List[Selection]] = [[], []]
        self.states: List[List[Tuple[torch.Tensor, torch.Tensor, torch.Tensor]]] = [[], []]
        self.acc, self.norms, self.unpacked = [], [], []
        for (n, m), k in zip(self.shapes, self.ks):
            for p in range(2):
                self.sels[p].append(Selection(m, k, dev))
                self.states[p].append(tuple(torch.empty(*_stored(layout, n, k), dtype=f32,
                                                        device=dev) for _ in range(3)))
            self.acc.append(torch.empty(*_stored(layout, n, m - k), dtype=f32, device=dev))
            self.norms.append(torch.empty(m, dtype=f32, device=dev))
            self.unpacked.append(torch.empty(*_stored(layout, n, m), dtype=f32, device=dev)
                                 if keep_unpacked else None)
        self.grad_slots = [list(s) for s in grad_slots]
        self.plans = [[self._plan(slot, p) for p in range(2)] for slot in range(len(self.grad_slots))]
        self.t = 0
        self.cur = 0

    def _plan(self, slot: int, p: int) -> Plan:
        q_bufs = []
        for q, ((n, m), k) in enumerate(zip(self.shapes, self.ks)):
            P, M, V = self.states[p][q]
            Pp, Mp, Vp = self.states[1 - p][q]
            src = StateSource(prev=self.sels[1 - p][q], prev_master=Pp, prev_exp_avg=Mp,
                              prev_exp_avg_sq=Vp,
                              init_master=self.init_master[q] if self.init_master else None)
            q_bufs.append(MatrixBuffers(
                grad=self.grad_slots[slot][q], k=k, sel=self.sels[p][q], weight=self.weights[q],
                master=P, exp_avg=M, exp_avg_sq=V, acc=self.acc[q], norms=self.norms[q],
                unpacked=self.unpacked[q], src=src, layout=self.layout))
        return Plan(q_bufs)

    @property
    def selection(self) -> List[Selection]:
        return self.sels[self.cur]

    @property
    def state(self):
        return self.states[self.cur]

    def step(self, stream=None, recorder=None) -> StepKind:
        """Enqueues one step (no synchronisation).  `recorder`, if given, is
        called as recorder(name) -> context manager around each launch (used
        to bracket launches with events on the launch stream)."""
        self.t += 1
        t = self.t
        kind = schedule(t, self.R, self.S)
        slot = (t - 1) % len(self.grad_slots)
        rec = recorder if recorder is not None else _no_record
        if kind.refresh:
            nxt = 0 if t == 1 else 1 - self.cur
            plan = self.plans[slot][nxt]
            with rec("colnorm"):
                plan.colnorm(stream)
            with rec("topk_select"):
                plan.topk_select(stream)
            mode = STATES_INIT if t == 1 else STATES_REMAP
            self.cur = nxt
        else:
            plan = self.plans[slot][self.cur]
            mode = STATES_INPLACE
        with rec("update_first" if kind.step_in_interval == 1 else "update"):
            plan.update(self.hp, t, mode, kind.step_in_interval, self.S, stream=stream)
        if kind.interval_end and self.keep_unpacked:
            with rec("unpack"):
                plan.unpack(1.0 / kind.step_in_interval, stream)
        return kind

    def close(self) -> None:
        for row in self.plans:
            for p in row:
                p.close()
