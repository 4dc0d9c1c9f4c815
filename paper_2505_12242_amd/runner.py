"""Per-step driver of the hot path over a set of weight matrices.

Owns the device buffers of every matrix (bf16 weight, compact fp32 states,
packed accumulation buffer, scores, selections, dense hand-over buffer) and
issues one batched launch per kernel per step:

    refresh step : zf_plan_colnorm -> zf_plan_topk_select ->
                   zf_plan_update (states remapped to the new selection)
    other steps  : zf_plan_update (states in place)
    interval end : zf_plan_update_handover, the update with the hand-over
                   fused in (out = (1/steps in the interval) x the final sums;
                   the packed buffer is only read), or zf_plan_update then
                   zf_plan_unpack when fuse_handover is False

Deferred packing (deferred_pack=True; either layout, fixed schedule, fused
hand-over): no packed buffer.  The unselected part of each step's gradient
stays in its gradient slot, every step but an interval's last runs the
Adam part alone, and the last step sums the interval's gradients (in step
order, the accumulation's own fp32 sequence) straight into the hand-over
(zf_plan_update_handover_deferred).  The slots must hold every gradient of
an interval: at least min(S, R) of them.  With Zen-auto decided on the
device (channel-major), every step sums the interval's kept gradients again
for the statistics and nothing is packed (zf_plan_update_zen_deferred,
zf_plan_handover_zen_deferred).

Compact states and selections are double-buffered: a refresh writes the new
selection and new states into the other buffer while reading the previous
ones (ZF_STATES_REMAP), so a column that stays selected carries its moments
without a separate pass.  Gradients come from caller-owned slots; step t
reads slot (t-1) mod len(slots).  Every tensor of the runner is stored in
one layout (ROW_MAJOR or CHANNEL_MAJOR, see the binding).

Zen-auto (zen_tau set; the adaptive interval of the paper's Zero-stall
Pipeline, "Hyperparameter Auto-tuning"): every update is zf_plan_update_zen,
which also measures the selected channels' gradient norms and the
accumulated channels' norms; the interval ends after the step whose pooled
mean accumulated norm reaches zen_tau times the pooled mean selected norm,
after `accum` (= S_max) steps, or before a refresh.  Without the offloaded
optimizer the decision stays on the device (zen_on_device, the default
there; both layouts): the update reads the interval's
position from a device state word, the totals kernel writes the end
decision into it, and a hand-over pass acts on it
(zf_plan_update_zen_device, zf_plan_handover_zen), so a step issues no
host synchronisation; the state and totals of each step are copied to
pinned host memory behind it and read only when the caller asks (the
returned step kind resolves lazily).  Otherwise the decision is taken on
the host from the 40-byte totals copied back after each update (one stream
synchronisation per step).

Offloaded optimizer (offload=True; Asynchronous Offloading Workflow and
Zero-stall Pipeline): every column's fp32 (p, m, v) lives in a full-state
store in pinned host memory.  A refresh swaps states against it inside the
update pass (columns entering the selection read their states from the
store, columns leaving write theirs back; the kernels access the pinned
store in place).  At every interval end the packed buffer is copied to the
host on a side stream and the deferred update (zf_host_adam_unselected, on
host threads, its own step counter) applies the interval's mean gradient to
the unselected columns of the store and produces their bf16 weights, which
zf_plan_scatter_weights writes into W.  With overlap=True the device
buffer is double-buffered, the copy and the host update run while the GPU
continues with the next interval, and the weights travel back to a device
staging buffer on the copy stream at the first step boundary after the host
finishes; the write-back kernel reads them there at the next boundary.
A refresh is the only step that reads the store.  Right after an interval
end (refresh_pending=True) it does not wait for the host: the interval's
host update starts once the refresh has read the store, and each column
entering the selection takes its owed step on the device first
(zf_plan_update_pending, from the still resident packed sums); the
write-back then leaves the refreshed selection's columns alone
(zf_plan_scatter_weights_skip_prev).  Otherwise a refresh waits for a
running host update.  Either way the results equal the synchronous order
bit for bit.
"""

from __future__ import annotations

import concurrent.futures
import os
import time
from dataclasses import dataclass
from typing import List, Optional, Sequence, Tuple

import numpy as np
import torch

from ._lib import (ROW_MAJOR, STATES_INIT, STATES_INPLACE, STATES_REMAP, ZEN_STATE_BYTES,
                   ZEN_TOTALS_BYTES, PinnedArena, copy_async,
                   AdamHparams, MatrixBuffers, Plan, Selection, StateSource, ZenTotals, _stored,
                   alloc_stored, padded_block,
                   host_adam_unselected, k_from_ratio)


@dataclass(frozen=True)
class StepKind:
    refresh: bool
    step_in_interval: int
    interval_end: bool


def schedule(t: int, R: int, S: int, warmup: int = 0) -> StepKind:
    """Refresh when (t-1) mod R == 0; an accumulation interval starts every S
    steps and at every refresh, and ends right before the next start.  The
    first `warmup` steps are synchronous (intervals of one step: the paper's
    warm-up without staleness); the S-step grid counts from step warmup + 1."""
    if t < 1 or R < 1 or S < 1 or warmup < 0:
        raise ValueError("t, R and S must be >= 1 and warmup >= 0")

    def last_start(x):
        if x <= warmup + 1:
            return x
        return max(x - (x - 1) % R, x - (x - warmup - 1) % S)

    start = last_start(t)
    nxt = t + 1
    end = nxt <= warmup + 1 or (nxt - 1) % R == 0 or (nxt - warmup - 1) % S == 0
    return StepKind(refresh=(t - 1) % R == 0, step_in_interval=t - start + 1, interval_end=end)


class DeviceZenStep:
    """The kind of a Zen-auto step whose interval the device decided: refresh
    is known on the host; the step's position in the interval, whether it
    ended the interval and the totals are read back from pinned host memory
    (after waiting for the step) the first time one of them is asked for."""

    def __init__(self, refresh: bool, host: torch.Tensor, event: torch.cuda.Event):
        self.refresh = refresh
        self._host = host
        self._event = event
        self._vals = None

    def resolve(self):
        if self._vals is None:
            self._event.synchronize()
            raw = self._host.numpy()
            # ended: 0, 1, or 2 when the update wrote the hand-over itself
            self._vals = (int(raw[0]), int(raw[1]), ZenTotals.from_bytes(raw[2:].tobytes()))
        return self._vals

    @property
    def fused(self) -> bool:
        """The step ended its interval and its update wrote the hand-over."""
        return self.resolve()[1] == 2

    @property
    def step_in_interval(self) -> int:
        return self.resolve()[0]

    @property
    def interval_end(self) -> bool:
        return self.resolve()[1] != 0

    @property
    def totals(self) -> ZenTotals:
        return self.resolve()[2]


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
                 device=None, keep_unpacked: bool = True, layout: int = ROW_MAJOR,
                 zen_tau: Optional[float] = None, offload: bool = False, overlap: bool = True,
                 host_threads: Optional[int] = None, fuse_handover: bool = True,
                 warmup: int = 0, refresh_pending: bool = True, first_step_stage: bool = True,
                 zen_on_device: bool = True, deferred_pack: bool = False):
        self.device = torch.device(device) if device is not None else torch.device("cuda")
        self.shapes = [(int(n), int(m)) for n, m in shapes]
        self.ratio, self.hp, self.R, self.S = ratio, hp, int(refresh), int(accum)
        self.warmup = int(warmup)
        self.ks = [k_from_ratio(ratio, m) for _, m in self.shapes]
        self.layout = layout
        self.offload = bool(offload)
        self.overlap = bool(overlap) and self.offload
        self.refresh_pending = bool(refresh_pending) and self.overlap
        self.keep_unpacked = keep_unpacked and not self.offload
        self.fuse_handover = bool(fuse_handover)
        # the bf16 first-step stage of the packed buffer (channel-major; the
        # fixed schedule with the fused hand-over, where the only consumers
        # of the packed buffer are the next update passes).  A refresh step
        # that starts an interval then fills it from the score pass.
        # (row-major: the fixed schedule with the fused hand-over only)
        # deferred packing (fixed schedule, hand-over fused, no offload): the
        # unselected part of every step's gradient stays in its slot until
        # the interval ends; the interval's last step sums them
        # (Zen-auto: decided on the device, channel-major; each step sums the
        # interval's kept gradients again for the statistics)
        self.deferred = bool(deferred_pack)
        if self.deferred:
            zen_ok = (zen_tau is None or (bool(zen_on_device) and layout != ROW_MAJOR))
            if not zen_ok or self.offload or not self.keep_unpacked or not self.fuse_handover:
                raise ValueError("deferred packing runs on the fixed schedule, or with Zen-auto "
                                 "decided on the device in the channel-major layout, with the "
                                 "fused hand-over, without offload")
            if len(grad_slots) < min(self.S, self.R):
                raise ValueError("deferred packing keeps every gradient of an interval: it needs "
                                 f"at least min(S, R) = {min(self.S, self.R)} gradient slots")
        self.use_stage = (bool(first_step_stage) and not self.offload and self.keep_unpacked
                          and not self.deferred
                          and (layout != ROW_MAJOR or (zen_tau is None and self.fuse_handover)))
        # with the fixed schedule and the fused hand-over a refresh step also
        # packs from the score pass: into the stage when an interval starts,
        # and (channel-major) into the hand-over buffer when the step is a
        # whole interval
        self.score_pack = self.use_stage and zen_tau is None and self.fuse_handover
        self.score_handover = ((self.score_pack or self.deferred) and layout != ROW_MAJOR
                               and zen_tau is None)
        self._in_stage = False  # the current interval's sums are in the stage
        self.weights = list(weights)
        self.init_master = list(init_master) if init_master is not None else None
        dev = self.device
        f32 = torch.float32
        self.zen_tau = None if zen_tau is None else float(zen_tau)
        # the interval decided on the device (no offload)
        self.zen_device = (self.zen_tau is not None and bool(zen_on_device)
                           and not self.offload)
        if self.zen_tau is not None:
            self.zen_totals = torch.zeros(ZEN_TOTALS_BYTES // 8, dtype=torch.int64, device=dev)
            self._zen_host = torch.zeros(ZEN_TOTALS_BYTES // 8, dtype=torch.int64,
                                         pin_memory=True)
            # device interval state {length, ended}: nothing accumulated yet
            self.zen_state = torch.tensor([0, 1], dtype=torch.int32, device=dev)
            assert self.zen_state.numel() * 4 == ZEN_STATE_BYTES
        self._last_totals: Optional[ZenTotals] = None
        self._zen_pending: Optional[DeviceZenStep] = None
        self._length = 0
        self._ended = True

        self.sels: List[List[Selection]] = [[], []]
        self.states: List[List[Tuple[torch.Tensor, torch.Tensor, torch.Tensor]]] = [[], []]
        nacc = 2 if self.overlap else 1
        self.accs: List[List[torch.Tensor]] = [[] for _ in range(nacc)]
        self.norms, self.unpacked, self.sel_sq, self.acc_sq = [], [], [], []
        self.store, self.host_acc, self.wcols, self.unsel_host = [], [], [], []
        # the offloaded optimizer's pinned host buffers: one exact-size arena
        self.arena = None
        if self.offload:
            total = 0
            for (n, m), k in zip(self.shapes, self.ks):
                full = (n, m) if layout == ROW_MAJOR else (m, n)
                total += 3 * PinnedArena.bytes_for(full, f32)
                total += PinnedArena.bytes_for(PinnedArena.stored_shape(layout, n, m - k, f32), f32)
                total += PinnedArena.bytes_for(
                    PinnedArena.stored_shape(layout, n, m - k, torch.bfloat16), torch.bfloat16)
                total += PinnedArena.bytes_for((m - k,), torch.int32)
            self.arena = PinnedArena(total)
        self.wcols_dev = []  # overlap: device staging of the host-produced weights
        self.stage = []      # bf16 first-step stage of the packed buffer
        for q, ((n, m), k) in enumerate(zip(self.shapes, self.ks)):
            if self.zen_tau is not None:
                self.sel_sq.append(torch.empty(k, dtype=f32, device=dev))
                self.acc_sq.append(torch.empty(m - k, dtype=f32, device=dev))
            for p in range(2):
                self.sels[p].append(Selection(m, k, dev))
                self.states[p].append(tuple(alloc_stored(layout, n, k, f32, dev)
                                            for _ in range(3)))
            for a in range(nacc):
                self.accs[a].append(None if self.deferred
                                    else alloc_stored(layout, n, m - k, f32, dev))
            if self.use_stage:
                self.stage.append(alloc_stored(layout, n, m, torch.bfloat16, dev))
            self.norms.append(torch.empty(m, dtype=f32, device=dev))
            self.unpacked.append(alloc_stored(layout, n, m, f32, dev)
                                 if self.keep_unpacked else None)
            if self.offload:
                p0 = (self.init_master[q] if self.init_master is not None
                      else self.weights[q].float())
                ar = self.arena
                sp = ar.take(p0.shape, f32)
                sp.copy_(p0)
                self.store.append((sp, ar.take(p0.shape, f32).zero_(),
                                   ar.take(p0.shape, f32).zero_()))
                self.host_acc.append(ar.take_stored(layout, n, m - k, f32))
                self.wcols.append(ar.take_stored(layout, n, m - k, torch.bfloat16))
                if self.overlap:
                    self.wcols_dev.append(alloc_stored(layout, n, m - k, torch.bfloat16, dev))
                self.unsel_host.append(self.arena.take((m - k,), torch.int32))
        self.grad_slots = [list(s) for s in grad_slots]
        self.plans = [[[self._plan(slot, p, a) for a in range(nacc)] for p in range(2)]
                      for slot in range(len(self.grad_slots))]
        self.t = 0
        self.cur = 0
        self.cur_a = 0
        # offloaded optimizer
        self.th = 0
        # default: the process's cores up to 16, one of them left to the
        # thread that keeps feeding the GPU while an overlapped update runs
        cores = min(16, len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity")
                    else (os.cpu_count() or 1))
        self.host_threads = (host_threads if host_threads is not None else
                             max(1, cores - 1) if self.overlap else cores)
        self._job: Optional[concurrent.futures.Future] = None
        self._job_p = 0         # selection buffer the running host update's interval used
        self._stg_p: Optional[int] = None  # same, for weights staged but not written back
        self._pend = None       # host update held back for the pending refresh
        self._ev_staged: Optional[torch.cuda.Event] = None
        self._ev_scatter: Optional[torch.cuda.Event] = None
        self._acc_free: List[Optional[torch.cuda.Event]] = [None] * nacc
        self._pool = (concurrent.futures.ThreadPoolExecutor(max_workers=1)
                      if self.overlap else None)
        self._copy_stream = torch.cuda.Stream(device=dev) if self.overlap else None
        self.pending_refreshes = 0  # refreshes that took over an unfinished host update
        self.stall_s = 0.0      # host time spent waiting for the deferred update
        self.host_update_s = 0.0  # host time inside the deferred update
        torch.cuda.synchronize(dev)  # store and host buffers ready before any kernel

    def _plan(self, slot: int, p: int, a: int) -> Plan:
        q_bufs = []
        for q, ((n, m), k) in enumerate(zip(self.shapes, self.ks)):
            P, M, V = self.states[p][q]
            Pp, Mp, Vp = self.states[1 - p][q]
            src = StateSource(prev=self.sels[1 - p][q], prev_master=Pp, prev_exp_avg=Mp,
                              prev_exp_avg_sq=Vp,
                              init_master=self.init_master[q] if self.init_master else None)
            if self.offload:
                src.store_master, src.store_exp_avg, src.store_exp_avg_sq = self.store[q]
            if self.refresh_pending:
                src.pend_acc = self.accs[1 - a][q]  # the interval before a refresh
            q_bufs.append(MatrixBuffers(
                grad=self.grad_slots[slot][q], k=k, sel=self.sels[p][q], weight=self.weights[q],
                master=P, exp_avg=M, exp_avg_sq=V, acc=self.accs[a][q], norms=self.norms[q],
                unpacked=self.unpacked[q], src=src, layout=self.layout,
                sel_sq=self.sel_sq[q] if self.sel_sq else None,
                acc_sq=self.acc_sq[q] if self.acc_sq else None,
                weight_cols=(self.wcols_dev[q] if self.overlap else self.wcols[q])
                if self.offload else None,
                acc_first=self.stage[q] if self.use_stage else None))
        return Plan(q_bufs)

    def _resolve_zen(self) -> None:
        """Zen-auto on the device: the host-side interval fields of the
        last step (position, end, whether its sums are in the stage, totals),
        read back now."""
        k = self._zen_pending
        if k is not None:
            length, end, tot = k.resolve()
            self._length, self._ended, self._last_totals = length, bool(end), tot
            # (a fused end writes the hand-over, not the stage)
            self._in_stage = self.use_stage and length == 1 and end != 2
            self._zen_pending = None

    @property
    def last_totals(self) -> Optional[ZenTotals]:
        self._resolve_zen()
        return self._last_totals

    @property
    def selection(self) -> List[Selection]:
        return self.sels[self.cur]

    @property
    def state(self):
        return self.states[self.cur]

    # ------------------------------------------------------------------ steps

    def step(self, stream=None, recorder=None) -> StepKind:
        """Enqueues one step.  Without Zen-auto or the offloaded optimizer the
        call does not synchronise.  `recorder`, if given, is called as
        recorder(name) -> context manager around each launch (used to
        bracket launches with events on the launch stream)."""
        st = stream if stream is not None else torch.cuda.current_stream(self.device)
        rec = recorder if recorder is not None else _no_record
        self.t += 1
        t = self.t
        if self.zen_tau is None:
            kind = schedule(t, self.R, self.S, self.warmup)
            refresh, length = kind.refresh, kind.step_in_interval
        elif self.zen_device:
            refresh = (t - 1) % self.R == 0
            length = None  # decided on the device
        else:
            refresh = (t - 1) % self.R == 0
            length = 1 if (refresh or self._ended or t <= self.warmup) else self._length + 1
            self._length = length
        if self.offload:
            self._before_step(refresh, length, st, rec)
        slot = (t - 1) % len(self.grad_slots)
        # a refresh with the stage: the score pass packs every channel (into
        # the stage when an interval starts; into the hand-over buffer when
        # the step is a whole interval) and the update only runs Adam
        staged = refresh and self.score_pack and not kind.interval_end
        scored_end = refresh and self.score_handover and kind.interval_end and length == 1
        if refresh:
            nxt = 0 if t == 1 else 1 - self.cur
            plan = self.plans[slot][nxt][self.cur_a]
            with rec("colnorm"):
                if staged:
                    plan.colnorm_stage(st)
                elif scored_end:
                    plan.colnorm_handover(1.0, st)
                else:
                    plan.colnorm(st)
            with rec("topk_select"):
                plan.topk_select(st)
            mode = STATES_INIT if t == 1 else STATES_REMAP
            self.cur = nxt
        else:
            plan = self.plans[slot][self.cur][self.cur_a]
            mode = STATES_INPLACE
        if self.zen_tau is None:
            end = kind.interval_end
            # an interval's first packed values sit in the stage, unless the
            # step handed over in the same pass (nothing packed then)
            self._in_stage = (self.use_stage and length == 1
                              and not (end and self.fuse_handover))
            if scored_end:
                with rec("update_adam_handover"):
                    plan.update_adam_handover(self.hp, t, mode, st)
                return kind
            if end and self.keep_unpacked and self.fuse_handover:
                if self.deferred and length > 1:
                    # the interval's earlier gradients, still in their slots
                    nsl = len(self.grad_slots)
                    earlier = [self.plans[(tt - 1) % nsl][self.cur][self.cur_a]
                               for tt in range(t - length + 1, t)]
                    with rec("update_handover"):
                        plan.update_handover_deferred(self.hp, t, earlier, 1.0 / length, st)
                else:
                    with rec("update_handover"):
                        plan.update_handover(self.hp, t, mode, length, self.S, 1.0 / length, st)
                return kind
            if refresh and self._pend is not None:
                scale_p, th_p = self._pend[:2]
                with rec("update_first"):
                    plan.update_pending(self.hp, t, self.S, th_p, scale_p, stream=st)
                self._start_held_update(st)
            else:
                adam_only = staged or self.deferred
                name = ("update_adam" if adam_only else "update_first" if length == 1
                        else "update_second" if length == 2 else "update")
                with rec(name):
                    plan.update(self.hp, t, mode, length, self.S, pack=not adam_only, stream=st)
        elif self.zen_device:
            # the interval ends on the device (trigger, S_max) or by the
            # caller's rule (before a refresh, warm-up steps); an end the
            # caller knows of is handed over by the update itself where the
            # plan can (force_end 2; the word then says ended = 2 and the
            # gated hand-over does nothing)
            force_end = (t % self.R == 0) or t <= self.warmup
            fuse = force_end and self.keep_unpacked and self.fuse_handover
            if self.deferred:
                # the plans of the steps an interval can still reach back to
                # (the device reads the last position - 1 of them)
                nsl = len(self.grad_slots)
                first = max(1, t - (min(self.S, self.R) - 1))
                earlier = [self.plans[(tt - 1) % nsl][self.cur][self.cur_a]
                           for tt in range(first, t)]
                with rec("update_zen"):
                    plan.update_zen_deferred(self.hp, t, mode, self.S, earlier,
                                             2 if fuse else int(force_end), self.zen_tau,
                                             self.zen_totals, self.zen_state, stream=st)
                with rec("handover_zen"):
                    plan.handover_zen_deferred(earlier, self.zen_state, st)
            else:
                with rec("update_zen"):
                    plan.update_zen_device(self.hp, t, mode, self.S,
                                           2 if fuse else int(force_end), self.zen_tau,
                                           self.zen_totals, self.zen_state, stream=st)
                if self.keep_unpacked:
                    with rec("handover_zen"):
                        plan.handover_zen(self.zen_state, st)
            host = torch.empty(2 + ZEN_TOTALS_BYTES // 4, dtype=torch.int32, pin_memory=True)
            with torch.cuda.stream(st):
                host[:2].copy_(self.zen_state, non_blocking=True)
                host[2:].copy_(self.zen_totals.view(torch.int32), non_blocking=True)
            ev = torch.cuda.Event()
            ev.record(st)
            kind = DeviceZenStep(refresh, host, ev)
            self._zen_pending = kind
            return kind
        else:
            if refresh and self._pend is not None:
                scale_p, th_p = self._pend[:2]
                with rec("update_zen_first"):
                    plan.update_zen_pending(self.hp, t, self.S, th_p, scale_p, self.zen_tau,
                                            self.zen_totals, stream=st)
                self._start_held_update(st)
            else:
                with rec("update_zen_first" if length == 1 else "update_zen"):
                    plan.update_zen(self.hp, t, mode, length, self.S, self.zen_tau,
                                    self.zen_totals, stream=st)
            with torch.cuda.stream(st):
                self._zen_host.copy_(self.zen_totals, non_blocking=True)
            st.synchronize()
            self._last_totals = ZenTotals.from_bytes(self._zen_host.numpy().tobytes())
            end = (self._last_totals.trigger or length >= self.S or t % self.R == 0
                   or t <= self.warmup)
            self._ended = end
            self._in_stage = self.use_stage and length == 1
            kind = StepKind(refresh=refresh, step_in_interval=length, interval_end=end)
        if end:
            if self.offload:
                self._hand_over(length, st, rec)
            elif self.keep_unpacked:
                with rec("unpack"):
                    if self.use_stage and length == 1:
                        plan.unpack_first(1.0, st)  # the sums are the stage's values
                    else:
                        plan.unpack(1.0 / length, st)
        return kind

    # --------------------------------------------------- offloaded optimizer

    def _start_held_update(self, st) -> None:
        """After a refresh that took over the entering columns' owed step:
        the held-back host update of the interval that just ended starts
        once the refresh has read the store."""
        scale_p, th_p, copied, p_old = self._pend
        self._pend = None
        swapped = torch.cuda.Event()
        swapped.record(st)
        self._job = self._pool.submit(self._host_update, scale_p, th_p, copied,
                                      self._ev_staged, swapped)
        self._job_p = p_old
        self.pending_refreshes += 1

    def _before_step(self, refresh: bool, length: int, st, rec) -> None:
        """Writes back weights staged at an earlier boundary, stages a
        finished host update (a refresh first waits for a running one: it
        reads the store), and makes a new interval wait until the device
        buffer it overwrites has been copied out."""
        if self._stg_p is not None:
            self._write_back(st, rec)
        if self._job is not None and (refresh or self._job.done()):
            self._finish_job(st, rec)
            if refresh and self._stg_p != self.cur:
                self._write_back(st, rec)  # its selection buffer is about to be refreshed
        if length == 1 and self._acc_free[self.cur_a] is not None:
            st.wait_event(self._acc_free[self.cur_a])
            self._acc_free[self.cur_a] = None

    def _finish_job(self, st, rec) -> None:
        """Waits for the running host update and stages its weights: with
        overlap, a copy to the device staging buffer on the copy stream."""
        t0 = time.perf_counter()
        self._job.result()
        self.stall_s += time.perf_counter() - t0
        self._job = None
        if self._stg_p is not None:
            self._write_back(st, rec)
        if self.overlap:
            cs = self._copy_stream
            if self._ev_scatter is not None:
                cs.wait_event(self._ev_scatter)  # the last write-back has read the staging buffer
            for q in range(len(self.shapes)):
                copy_async(padded_block(self.wcols_dev[q]), padded_block(self.wcols[q]), cs)
            ev = torch.cuda.Event()
            ev.record(cs)
            self._ev_staged = ev
        self._stg_p = self._job_p

    def _write_back(self, st, rec) -> None:
        """W[:, unsel] = the staged weights, under the selection their
        interval used; after a refresh the refreshed selection's columns are
        left alone (they belong to the selective optimizer)."""
        p = self._stg_p
        if self.overlap:
            st.wait_event(self._ev_staged)
        plan = self.plans[0][p][0]
        with rec("scatter_weights"):
            if p == self.cur:
                plan.scatter_weights(st)
            else:
                plan.scatter_weights_skip_prev(st)
        ev = torch.cuda.Event()
        ev.record(st)
        self._ev_scatter = ev
        self._stg_p = None

    def _host_update(self, scale: float, th: int, copied, *waits) -> None:
        """The deferred update of every matrix on the host threads.  copied:
        one event (or one per matrix) after which the packed sums are on the
        host; waits: the previous staging copy has read the weight columns,
        the refresh has read the store."""
        for ev in waits:
            if ev is not None:
                ev.synchronize()
        per = copied if isinstance(copied, list) else [copied] * len(self.shapes)
        t0 = time.perf_counter()
        for q, ((n, m), k) in enumerate(zip(self.shapes, self.ks)):
            if per[q] is not None:
                per[q].synchronize()
            P, M, V = self.store[q]
            host_adam_unselected(self.host_acc[q], self.unsel_host[q], n, m, k, scale, P, M, V,
                                 self.wcols[q], self.hp, th, layout=self.layout,
                                 nthreads=self.host_threads)
        self.host_update_s += time.perf_counter() - t0

    def _hand_over(self, length: int, st, rec) -> None:
        self.th += 1
        scale = float(np.float32(1.0 / length))
        a = self.cur_a
        sels = self.sels[self.cur]
        if not self.overlap:
            for q in range(len(self.shapes)):
                copy_async(padded_block(self.host_acc[q]), padded_block(self.accs[a][q]), st)
                copy_async(self.unsel_host[q], sels[q].unsel_idx, st)
            st.synchronize()
            self._host_update(scale, self.th, None)
            self._stg_p = self.cur
            self._write_back(st, rec)
            return
        if self._job is not None:  # the host is still busy with the previous interval
            self._finish_job(st, rec)
        ev = torch.cuda.Event()
        ev.record(st)
        cs = self._copy_stream
        cs.wait_event(ev)
        # one event per matrix: the host update starts on a matrix as soon as
        # its sums have arrived, while the later ones still copy
        copied = []
        for q in range(len(self.shapes)):
            copy_async(self.unsel_host[q], sels[q].unsel_idx, cs)
            copy_async(padded_block(self.host_acc[q]), padded_block(self.accs[a][q]), cs)
            e = torch.cuda.Event()
            e.record(cs)
            copied.append(e)
        self._acc_free[a] = copied[-1] if copied else None
        warm = self.t <= self.warmup
        if self.refresh_pending and not warm and self.t % self.R == 0:
            # the next step refreshes: it takes over the columns entering its
            # selection and then starts this host update (see step)
            self._pend = (scale, self.th, copied, self.cur)
        else:
            self._job = self._pool.submit(self._host_update, scale, self.th, copied,
                                          self._ev_staged)
            self._job_p = self.cur
        self.cur_a = 1 - a
        if warm:
            # warm-up: synchronous, the update lands before the next step
            self._finish_job(st, rec)
            self._write_back(st, rec)

    def sync(self, stream=None) -> None:
        """Finishes every outstanding deferred update and write-back and
        synchronises the device (the state the synchronous order reaches)."""
        st = stream if stream is not None else torch.cuda.current_stream(self.device)
        if self._pend is not None:
            # no refresh took the held-back update over: run it as usual
            scale_p, th_p, copied, p = self._pend
            self._pend = None
            self._job = self._pool.submit(self._host_update, scale_p, th_p, copied,
                                          self._ev_staged)
            self._job_p = p
        if self._job is not None:
            self._finish_job(st, _no_record)
        if self._stg_p is not None:
            self._write_back(st, _no_record)
        torch.cuda.synchronize(self.device)

    # ---------------------------------------------------- checkpoint / resume

    def state_dict(self) -> dict:
        """What a later run needs to continue bit for bit: the step
        counters, the current selection and compact states, the current
        interval's packed sums and, with the offloaded optimizer, the store
        and its step counter.  Drains the pipeline first (sync).  Tensors are
        CPU copies in the runner's layout; the weights stay the caller's."""
        if self.deferred:
            raise NotImplementedError("deferred packing keeps an interval's sums in the "
                                      "gradient slots: no checkpoint of them")
        self.sync()
        self._resolve_zen()
        c, a = self.cur, self.cur_a
        mats = []
        for q in range(len(self.shapes)):
            s = self.sels[c][q]
            d = {"sel_idx": s.sel_idx.cpu(), "unsel_idx": s.unsel_idx.cpu(),
                 "mask": s.mask.cpu(), "prefix": s.prefix.cpu(),
                 "master": self.states[c][q][0].cpu(), "exp_avg": self.states[c][q][1].cpu(),
                 "exp_avg_sq": self.states[c][q][2].cpu(), "acc": self.acc[q].cpu()}
            if self.offload:
                d["store"] = [x.clone() for x in self.store[q]]
            mats.append(d)
        return {"shapes": list(self.shapes), "ks": list(self.ks), "layout": self.layout,
                "R": self.R, "S": self.S, "warmup": self.warmup, "zen_tau": self.zen_tau,
                "offload": self.offload, "t": self.t, "th": self.th, "length": self._length,
                "ended": self._ended, "in_stage": self._in_stage, "mats": mats}

    def load_state_dict(self, sd: dict) -> None:
        """Continues from a state_dict of a runner with the same shapes,
        ratio, layout, schedule and offload mode (the caller restores the
        weights)."""
        if self.deferred:
            raise NotImplementedError("deferred packing keeps an interval's sums in the "
                                      "gradient slots: no checkpoint of them")
        mine = {"shapes": list(self.shapes), "ks": list(self.ks), "layout": self.layout,
                "R": self.R, "S": self.S, "warmup": self.warmup, "zen_tau": self.zen_tau,
                "offload": self.offload}
        for key, val in mine.items():
            got = [tuple(x) for x in sd[key]] if key == "shapes" else sd[key]
            want = [tuple(x) for x in val] if key == "shapes" else val
            if got != want:
                raise ValueError(f"state_dict {key} = {sd[key]!r}, this runner has {val!r}")
        self.sync()
        self.cur, self.cur_a = 0, 0
        # the next step is an interval's second: with the stage it reads the
        # first step's values there, whichever runner saved them
        t_saved = int(sd["t"])
        if self.zen_tau is None:
            k = schedule(t_saved, self.R, self.S, self.warmup) if t_saved >= 1 else None
            first_only = k is not None and k.step_in_interval == 1 and not k.interval_end
        else:
            first_only = int(sd["length"]) == 1 and not bool(sd["ended"])
        to_stage = self.use_stage and (bool(sd.get("in_stage")) or first_only)
        for q, d in enumerate(sd["mats"]):
            s = self.sels[0][q]
            for dst, key in ((s.sel_idx, "sel_idx"), (s.unsel_idx, "unsel_idx"),
                             (s.mask, "mask"), (s.prefix, "prefix")):
                dst.copy_(d[key])
            for dst, key in zip(self.states[0][q], ("master", "exp_avg", "exp_avg_sq")):
                dst.copy_(d[key])
            if to_stage:
                # first-step values (exact in bf16) into the unselected rows
                self.stage[q].index_copy_(1 if self.layout == ROW_MAJOR else 0,
                                          s.unsel_idx.long(),
                                          d["acc"].to(self.device, torch.bfloat16))
            self.accs[0][q].copy_(d["acc"])
            if self.offload:
                for dst, src in zip(self.store[q], d["store"]):
                    dst.copy_(src)
        self.t, self.th = int(sd["t"]), int(sd["th"])
        self._length, self._ended = int(sd["length"]), bool(sd["ended"])
        self._in_stage = to_stage
        self._zen_pending = None
        if self.zen_tau is not None:
            self.zen_state.copy_(torch.tensor([self._length, int(self._ended)], dtype=torch.int32))
        self._acc_free = [None] * len(self._acc_free)
        torch.cuda.synchronize(self.device)

    @property
    def acc(self) -> List[torch.Tensor]:
        """The last interval's packed sums, fp32 (after an interval's first
        step with the bf16 stage: a widened copy of the stage, exact)."""
        if self.deferred:
            raise AttributeError("deferred packing materialises no packed buffer")
        self._resolve_zen()
        if self._in_stage:
            dim = 1 if self.layout == ROW_MAJOR else 0
            return [x.index_select(dim, s.unsel_idx.long()).float()
                    for x, s in zip(self.stage, self.sels[self.cur])]
        return self.accs[self.cur_a]

    @property
    def current_acc(self) -> List[torch.Tensor]:
        """The fp32 packed buffers of the current interval (double-buffered
        when the deferred update overlaps); after an interval's first step
        with the bf16 stage the sums are in the stage (see acc)."""
        return self.accs[self.cur_a]

    def close(self) -> None:
        if self._job is not None:
            self._job.result()
            self._job = None
        self._pend = None
        if self._pool is not None:
            self._pool.shutdown(wait=True)
        for row in self.plans:
            for pp in row:
                for plan in pp:
                    plan.close()  # (synchronises the device)
        if self.arena is not None:
            # the store and staging tensors live in the arena: invalid from here on
            self.store, self.host_acc, self.wcols, self.unsel_host = [], [], [], []
            self.arena.free()
            self.arena = None
