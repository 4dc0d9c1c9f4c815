#!/usr/bin/env python3
"""Throughput of the selective-update hot path on one MI355X.

Workload (default): the full Llama-2-7B-shaped gradient set -- embedding,
32 decoder layers (q/k/v/o 4096x4096, gate/up 11008x4096, down 4096x11008)
and LM head, 226 matrices, 6,738,149,376 parameters -- with bf16 gradients
(lognormal(0, 1.5) column scales, 5% temporal jitter), fp32 compact Adam
states, top-k ratio 10%, selection refresh R = 4 and accumulation interval
S = 4.  Gradients live in a ring of device buffers generated before timing
(step t reads slot (t-1) mod slots), so every input is resident in HBM when
the timed region starts.

A step is one pass of the whole hot path over the set: on refresh steps
column scores + top-k, then the fused Adam/pack pass (states remapped on
refresh), and on interval ends the dense hand-over (unpack).  Warm-up steps
are untimed; the timed steps are bracketed by device synchronisation.

Prints one JSON line: algorithmic GB/s (value), fraction of the 8 TB/s HBM
peak, params/s, per-kernel times, the roofline of the dominant kernel
(the fused Adam/pack pass) and the CPU oracle timed on a bounded sample.
"""

from __future__ import annotations

import argparse
import contextlib
import gc
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
HBM_PEAK_GBS = 8000.0  # MI355X HBM3E, published
PROFILES = os.path.join(ROOT, "profiles")
# Zen-auto with deferred packing reads 2p bytes per unselected element at the
# interval's step p: p(p + 1) + 4 bytes over an interval of p steps ended by
# force, against 10p - 8 packing every step with the bf16 stage.  Measured on
# MI355X: 10.0-10.3 against 11.6-11.7 ms per 7B step at 4 steps, 16.8-17.0
# against 15.5-15.6 ms for the 70B share at 8 steps.
ZEN_DEFER_MAX = 6

KERNEL_SOURCES = [os.path.join(ROOT, "paper_2505_12242_amd", "csrc", f)
                  for f in ("zf_device.hpp", "zf_internal.hpp", "zf_kernels.hip",
                            "zf_kernels_cm.hip", "zf_kernels_rv.hip", "zf_kernels_stream.hip")]


def parse_args(argv=None):
    ap = argparse.ArgumentParser(description=__doc__.split("\n\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=16)
    ap.add_argument("--warmup", type=int, default=16)
    ap.add_argument("--workload", default="llama2-7b-full")
    ap.add_argument("--slots", type=int, default=3, help="gradient buffers in the ring")
    ap.add_argument("--layout", choices=["channel-major", "row-major"], default="channel-major",
                    help="storage of every matrix: channel-major (each input channel one "
                         "contiguous row, the paper's column-major gradient storage) or "
                         "PyTorch's row-major [out, in]")
    ap.add_argument("--layers", type=int, default=None,
                    help="keep only the first N decoder layers of the workload (with its "
                         "embedding and LM head), e.g. the part of a set whose offloaded "
                         "optimizer fits the pinned host memory")
    ap.add_argument("--ratio", type=float, default=None, help="override the top-k ratio")
    ap.add_argument("--refresh", type=int, default=None, help="override the refresh interval R")
    ap.add_argument("--accum", type=int, default=None, help="override the accumulation interval S")
    ap.add_argument("--zen-tau", type=float, default=None,
                    help="run Zen-auto (adaptive interval, at most --accum steps) with this "
                         "threshold instead of the fixed schedule")
    ap.add_argument("--zen-on-host", action="store_true",
                    help="with --zen-tau: decide each interval end on the host (one stream "
                         "synchronisation per step) instead of on the device")
    ap.add_argument("--offload", action="store_true",
                    help="run the whole method with offloaded optimizer states: full-state "
                         "store in pinned host memory (swapped at refreshes) and the deferred "
                         "host update of the unselected columns at every interval end, "
                         "overlapped with the following steps")
    ap.add_argument("--no-overlap", action="store_true",
                    help="with --offload: run the deferred update synchronously")
    ap.add_argument("--no-first-step-stage", action="store_true",
                    help="keep an interval's first packed values in fp32 (default: a bf16 "
                         "stage, 2 B per value written and read)")
    ap.add_argument("--refresh-waits", action="store_true",
                    help="with --offload: a refresh right after an interval end waits for the "
                         "host update (default: the device takes over the entering columns)")
    ap.add_argument("--model-compute-ms", type=float, default=0.0,
                    help="with --offload: before every step, this much stand-in model compute on "
                         "the GPU (bf16 matrix products on the step's stream), for the forward and "
                         "backward passes that the deferred host update overlaps with")
    ap.add_argument("--host-threads", type=int, default=None,
                    help="with --offload: host threads of the deferred update (default: "
                         "min(16, cpu count))")
    ap.add_argument("--packing", choices=["deferred", "every-step"], default=None,
                    help="deferred (default where it applies: fixed schedule, or Zen-auto "
                         "decided on the device in the channel-major layout with intervals of "
                         "at most 6 steps; fused hand-over, no offload): every gradient of an "
                         "interval stays in its slot and the interval's last step sums them "
                         "into the hand-over (Zen-auto: every step sums them for its "
                         "statistics), with no packed buffer (the ring gets at least min(S, R) "
                         "slots); every-step: the unselected part is accumulated into the "
                         "packed buffer at every step")
    ap.add_argument("--separate-handover", action="store_true",
                    help="hand over with a separate unpack pass after the last update of an "
                         "interval instead of fusing it into that update")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample", choices=["set", "layer"], default="set",
                    help="matrices the all-core oracle timing covers: the whole set, or the "
                         "first decoder layer (the one-thread timing always covers that layer)")
    ap.add_argument("--cpu-sample-steps", type=int, default=4)
    ap.add_argument("--calibration-gib", type=float, default=8.0,
                    help="size of the reference streams (read, copy, read-modify-write) timed "
                         "before the workload; the copy is also the PMC calibration point "
                         "(0: skip)")
    return ap.parse_args(argv)


# ---------------------------------------------------------------------------
# byte model: the bytes each kernel must move, per matrix
# ---------------------------------------------------------------------------

def step_traffic(shapes, ks, refresh: bool, first: bool, end: bool, offload: bool = False,
                 fused_handover: bool = False, second: bool = False, stage: bool = False,
                 scored_handover: bool = None, deferred: bool = False, length: int = 1,
                 zen: bool = False) -> dict:
    """Algorithmic HBM bytes of one step, by kernel, as [read, written].

    colnorm  2nm (read G) + 4m (write scores)          refresh steps
    topk     4m (read scores) + 4m (write indices)
             + 12 ceil(m/64) (mask and prefix)         refresh steps
    update   28nk: per selected element G 2 + P/M/V 12 read + 12 write + W 2;
             6nu / 10nu: per unselected element G 2 + A 4 write (+ A 4 read
             after the interval's first step)
    unpack   4nu (read A) + 4nm (write the dense buffer)  interval ends
             offloaded optimizer instead: 4nu (A read by the device -> host
             copy) + 2nu (bf16 weights written back by the scatter)
             fused into the update (the interval's last step): the update
             writes the hand-over instead of A -- the same 10nu (6nu) for the
             unselected part -- plus 4nk zeros at the selected columns; A is
             neither written nor read back
    stage    with the bf16 first-step stage of A (channel-major): an
             interval's first step writes 2 B per unselected element
             instead of 4 (4nu instead of 6nu; 6nu when it also hands over
             in the same pass, as before) and its second step reads 2 B
             instead of 4 (8nu instead of 10nu); a separate hand-over pass
             after a one-step interval reads the stage (2nu instead of 4nu).
             With the fused hand-over a refresh step that starts an
             interval fills the stage from the score pass instead: colnorm
             2nm + 2nm (every channel's row written), update 28nk (Adam
             only); a refresh step that is a whole (one-step) interval takes
             its hand-over from the score pass (scored_handover, channel-
             major; default: with the stage): colnorm 2nm + 4nm, update
             28nk + 4nk (the selected rows' zeros)
    deferred packing (deferred; fused hand-over): no packed buffer.  Every
             step but an interval's last updates the selected part only
             (28nk); the last, of `length` >= 2 steps, reads each step's
             gradient once at the unselected elements and writes the
             hand-over: 28nk + 4nk + (2 length + 4) nu.  One-step intervals
             as with the stage (the score pass hands over on a refresh)
    Zen-auto with deferred packing (deferred and zen): every step, at
             position `length` in its interval, reads the interval's kept
             gradients at the unselected elements for the statistics
             (28nk + 2 length nu); an end the caller forces writes the
             hand-over from the update (+ 4nu + 4nk), any other end from the
             gated hand-over pass (unpack: 2 length nu + 4nm)
    """
    if scored_handover is None:
        scored_handover = stage or deferred
    out = {"colnorm": [0, 0], "topk_select": [0, 0], "update": [0, 0], "unpack": [0, 0]}

    def add(cls, r, w):
        out[cls][0] += r
        out[cls][1] += w

    for (n, m), k in zip(shapes, ks):
        u = m - k
        staged_refresh = refresh and stage and fused_handover and not end
        scored_end = refresh and scored_handover and fused_handover and end and first
        if refresh:
            add("colnorm", 2 * n * m, 4 * m + (2 * n * m if staged_refresh else 0)
                + (4 * n * m if scored_end else 0))
            add("topk_select", 4 * m, 4 * m + 12 * ((m + 63) // 64))
        # selected: G 2 + P/M/V 12 read, P/M/V 12 + W 2 written
        add("update", 14 * n * k, 14 * n * k)
        if deferred and zen:
            add("update", 2 * length * n * u, 0)
            if end:
                if fused_handover:
                    add("update", 0, 4 * n * u + 4 * n * k)
                else:
                    add("unpack", 2 * length * n * u, 4 * n * m)
            continue
        if deferred and not scored_end and not (end and first):
            if end:  # each step's gradient read once, the hand-over written
                add("update", 2 * length * n * u, 4 * n * u + 4 * n * k)
            continue
        if staged_refresh or scored_end:
            pass  # the score pass did the packing
        elif first:
            # G read; the fused hand-over of a one-step interval writes no
            # packed values (it writes the hand-over: 4)
            add("update", 2 * n * u, (2 if (stage and not (end and fused_handover)) else 4) * n * u)
        else:
            # G and the previous sums (the stage's 2 B on the second step) read, 4 written
            add("update", (4 if (stage and second) else 6) * n * u, 4 * n * u)
        if end:
            if offload:
                add("unpack", 4 * n * u, 2 * n * u)
            elif fused_handover:
                add("update", 0, 4 * n * k)
            else:
                # the separate pass reads the stage after a one-step interval
                add("unpack", (2 if (stage and first) else 4) * n * u, 4 * n * m)
    return out


def step_bytes(shapes, ks, refresh: bool, first: bool, end: bool, offload: bool = False,
               fused_handover: bool = False, second: bool = False, stage: bool = False,
               scored_handover: bool = None, deferred: bool = False, length: int = 1,
               zen: bool = False) -> dict:
    """step_traffic's bytes read + written, by kernel."""
    t = step_traffic(shapes, ks, refresh, first, end, offload, fused_handover, second, stage,
                     scored_handover, deferred, length, zen)
    return {cls: r + w for cls, (r, w) in t.items()}


# ---------------------------------------------------------------------------
# device-resident synthetic gradient set
# ---------------------------------------------------------------------------

def build_set(wl, slots: int, device, layout: int = 0):
    """Gradient ring and bf16 weights of workload wl on the device, stored in
    `layout` (channel-major tensors are the transposes of the logical
    [out, in] matrices)."""
    import torch
    from workloads import derive_seed, gradient, master_weights, step_scales
    import paper_2505_12242_amd as zf

    def store(x):
        return x if layout == zf.ROW_MAJOR else x.t().contiguous()

    shapes = [(mt.n, mt.m) for mt in wl.matrices]
    ks = [zf.k_from_ratio(wl.ratio, m) for _, m in shapes]
    grad_slots = []
    for s in range(slots):
        t = s + 1
        buf = []
        for q, (n, m) in enumerate(shapes):
            sc = step_scales(wl, q, t, k_boundary=ks[q])
            buf.append(store(gradient(n, m, sc, derive_seed(wl.seed, q, "grad", t),
                                      device=device)))
        grad_slots.append(buf)
    weights = []
    for q, (n, m) in enumerate(shapes):
        w = master_weights(n, m, derive_seed(wl.seed, q, "master"), wl.master_std, device=device)
        weights.append(store(w.to(torch.bfloat16)))
        del w
    return shapes, ks, grad_slots, weights


# ---------------------------------------------------------------------------
# CPU oracle baseline on a bounded sample
# ---------------------------------------------------------------------------

def host_info() -> dict:
    """The host the oracle is timed on: usable cores, CPU model, sockets /
    NUMA nodes, memory."""
    info = {"nproc": len(os.sched_getaffinity(0)), "cpu_count": os.cpu_count()}
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    info["model"] = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        import subprocess
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in out.splitlines():
            key, _, val = line.partition(":")
            if key.strip() in ("Socket(s)", "NUMA node(s)", "Thread(s) per core",
                               "Core(s) per socket"):
                info[key.strip()] = val.strip()
    except Exception:
        pass
    try:
        with open("/proc/meminfo") as f:
            info["mem_GB"] = round(int(f.readline().split()[1]) * 1024 / 1e9, 1)
    except (OSError, ValueError, IndexError):
        pass
    return info


def _oracle_worker(conn) -> None:
    """One process of the all-core oracle timing (spawned: no torch, no GPU).
    Receives its matrices' jobs (shared-memory names of the initial bf16
    weight and of the gradients, the step -> gradient map, the workload's
    hyperparameters), builds one oracle per matrix, reports ready, and on
    "go" runs the steps, timing them with the system-wide monotonic clock."""
    import hashlib as _hl
    from multiprocessing import shared_memory

    import numpy as np
    import oracle as O

    jobs = conn.recv()
    held, work = [], []
    for job in jobs:
        n, m = job["shape"]

        def view(name):
            shm = shared_memory.SharedMemory(name=name)
            held.append(shm)
            return np.ndarray((n, m), dtype=np.uint16, buffer=shm.buf)

        W = view(job["w"])
        G = [view(x) for x in job["g"]]
        orc = O.MatrixOracle(O.widen(W), W, job["ratio"], *job["hyper"], job["R"], job["S"])
        work.append((orc, G, job["slots"]))
    conn.send("ready")
    conn.recv()
    t0 = time.monotonic()
    for t in range(len(work[0][2]) if work else 0):
        for orc, G, slots in work:
            orc.step(G[slots[t]])
    t1 = time.monotonic()
    digests = [_hl.sha256(orc.P.tobytes() + orc.W.tobytes() + orc.A.tobytes()).hexdigest()[:16]
               for orc, _, _ in work]
    del work
    for shm in held:
        shm.close()
    conn.send({"start": t0, "end": t1, "digests": digests})


class HostSample:
    """The oracle's inputs for the CPU baseline in shared memory (logical
    [out, in] bf16 bits): every sampled matrix's initial weight, copied
    before the GPU run changes it, and the gradients its steps read."""

    def __init__(self, wl, qs, weights, layout: int):
        from multiprocessing import shared_memory

        import numpy as np
        import torch
        self.qs = list(qs)
        self.shm = {}
        self.layout = layout
        self._np = np
        self._shared_memory = shared_memory
        for q in self.qs:
            self.shm[("w", q)] = self._put(weights[q], torch)

    def _put(self, t, torch):
        x = t if self.layout == 0 else t.t()
        n, m = x.shape
        shm = self._shared_memory.SharedMemory(create=True, size=max(1, n * m * 2))
        host = torch.from_numpy(self._np.ndarray((n, m), dtype=self._np.int16, buffer=shm.buf))
        host.copy_(x.view(torch.int16))
        return shm

    def add_grads(self, grad_slots, steps: int):
        """The gradients steps 1..steps read (step t reads ring slot
        (t-1) mod len(grad_slots), as on the device)."""
        import torch
        ring = len(grad_slots)
        self.steps = steps
        self.used = sorted({(t - 1) % ring for t in range(1, steps + 1)})
        self.step_slot = [self.used.index((t - 1) % ring) for t in range(1, steps + 1)]
        for q in self.qs:
            for s in self.used:
                self.shm[("g", q, s)] = self._put(grad_slots[s][q], torch)

    def array(self, key, shape):
        return self._np.ndarray(shape, dtype=self._np.uint16, buffer=self.shm[key].buf)

    def close(self):
        for shm in self.shm.values():
            shm.close()
            shm.unlink()
        self.shm = {}


def cpu_baseline(wl, shapes, ks, sample: "HostSample", one_thread_qs, workers: int) -> dict:
    """Times the oracle (as it stands) on the host over the sample's steps
    1..steps of the workload's schedule:
      one thread -- the matrices one_thread_qs in this process;
      all cores  -- every sampled matrix, one process per core (matrices
                    assigned longest first), all starting together; the
                    wall time runs from the first start to the last end.
    Each matrix's oracle is independent and deterministic, so the all-core
    run gives the same results as one thread; the digests of the
    one-thread matrices' final states are compared to show it."""
    import hashlib as _hl

    import oracle as O
    hp = wl.hyper
    hyper = (hp.lr, hp.beta1, hp.beta2, hp.eps, hp.weight_decay)
    steps = sample.steps
    slots = sample.step_slot  # step t (0-based) -> index into sample.used

    def sample_bytes(qs):
        total = 0
        for q in qs:
            for t in range(1, steps + 1):
                kind = O.schedule(t, wl.refresh, wl.accum)
                total += sum(step_bytes([shapes[q]], [ks[q]], kind.refresh,
                                        kind.step_in_interval == 1, kind.interval_end).values())
        return total

    # one thread, in this process
    elapsed = 0.0
    digests1 = {}
    for q in one_thread_qs:
        n, m = shapes[q]
        W = sample.array(("w", q), (n, m))
        orc = O.MatrixOracle(O.widen(W), W, wl.ratio, *hyper, wl.refresh, wl.accum)
        G = [sample.array(("g", q, s), (n, m)) for s in sample.used]
        for t in range(steps):
            t0 = time.perf_counter()
            orc.step(G[slots[t]])
            elapsed += time.perf_counter() - t0
        digests1[q] = _hl.sha256(orc.P.tobytes() + orc.W.tobytes() + orc.A.tobytes()).hexdigest()[:16]
        del orc, G, W
    b1 = sample_bytes(one_thread_qs)
    p1 = sum(shapes[q][0] * shapes[q][1] for q in one_thread_qs)
    out = {
        "one_thread": {"GB/s": round(b1 / elapsed / 1e9, 4),
                       "params_per_s": round(p1 * steps / elapsed, 1),
                       "seconds": round(elapsed, 3),
                       "sample": f"{len(one_thread_qs)} matrices ({p1:,} params), steps 1-{steps}"},
    }

    try:
        out["all_cores"] = _all_cores(wl, shapes, ks, sample, workers, hyper, slots,
                                      sample_bytes, digests1)
    except Exception as e:  # the one-thread figure stands; say why
        out["all_cores_error"] = f"{type(e).__name__}: {e}"
    return out


def _all_cores(wl, shapes, ks, sample, workers, hyper, slots, sample_bytes, digests1) -> dict:
    """The all-core leg of cpu_baseline: one spawned process per core."""
    import multiprocessing as mp
    steps = sample.steps
    qs = sorted(sample.qs, key=lambda q: -shapes[q][0] * shapes[q][1])
    nw = max(1, min(workers, len(qs)))
    assign = [[] for _ in range(nw)]
    load = [0] * nw
    for q in qs:
        w = load.index(min(load))
        assign[w].append(q)
        load[w] += shapes[q][0] * shapes[q][1]
    ctx = mp.get_context("spawn")
    saved = {k: os.environ.get(k) for k in ("OMP_NUM_THREADS", "OPENBLAS_NUM_THREADS",
                                            "MKL_NUM_THREADS")}
    for k in saved:
        os.environ[k] = "1"
    procs, conns = [], []
    try:
        for w in range(nw):
            a, b = ctx.Pipe()
            p = ctx.Process(target=_oracle_worker, args=(b,), daemon=True)
            p.start()
            procs.append(p)
            conns.append(a)
    finally:
        for k, v in saved.items():
            if v is None:
                os.environ.pop(k, None)
            else:
                os.environ[k] = v
    for w in range(nw):
        conns[w].send([{"shape": shapes[q], "w": sample.shm[("w", q)].name,
                        "g": [sample.shm[("g", q, s)].name for s in sample.used],
                        "slots": slots, "ratio": wl.ratio, "hyper": hyper, "R": wl.refresh,
                        "S": wl.accum} for q in assign[w]])
    def receive(c, timeout):
        if not c.poll(timeout):
            raise TimeoutError("an oracle process did not answer")
        return c.recv()

    try:
        for c in conns:
            if receive(c, 600) != "ready":
                raise RuntimeError("an oracle process failed to start")
        for c in conns:
            c.send("go")
        res = [receive(c, 1800) for c in conns]
    finally:
        for p in procs:
            p.join(timeout=60)
            if p.is_alive():
                p.kill()
    wall = max(r["end"] for r in res) - min(r["start"] for r in res)
    digests = {q: d for w, r in enumerate(res) for q, d in zip(assign[w], r["digests"])}
    ball = sample_bytes(sample.qs)
    pall = sum(shapes[q][0] * shapes[q][1] for q in sample.qs)
    return {
        "GB/s": round(ball / wall / 1e9, 4),
        "params_per_s": round(pall * steps / wall, 1),
        "seconds": round(wall, 3),
        "processes": nw,
        "sample": f"{len(sample.qs)} matrices ({pall:,} params), steps 1-{steps}",
        "same_results_as_one_thread": all(digests.get(q) == d for q, d in digests1.items()),
    }


# ---------------------------------------------------------------------------
# PMC traffic recorded for the current kernel source
# ---------------------------------------------------------------------------

def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for path in KERNEL_SOURCES:
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def launch_kernels(kind: str, channel_major: bool, deferred: bool, stage: bool = False,
                   scored_handover: bool = False) -> str:
    """The kernels behind one launch kind of the runner."""
    if kind == "colnorm":
        what = ("column scores, and every channel's hand-over of the one-step interval"
                if scored_handover else "column scores, and the bf16 first-step stage"
                if stage else "column scores")
        return (f"cm_colnorm_kernel ({what})" if channel_major else
                f"colnorm_partial_kernel + colnorm_finalize_kernel ({what})")
    if channel_major and kind == "update_adam_handover":
        return ("cm_update_kernel, selected-only grid (Adam + bf16 write-back, +0.0 in the "
                "selected channels' hand-over rows)")
    if channel_major:
        if deferred and kind == "update_zen":
            return ("cm_update_kernel, Zen-auto with deferred packing (Adam + statistics of the "
                    "interval's running sum, summed from the kept gradients)")
        if deferred and kind == "update_handover":
            return ("cm_handover_deferred_kernel (the interval's last step: Adam + the sum of "
                    "the interval's gradients into the hand-over)")
        if kind == "update_adam":
            return "cm_update_kernel, selected-only grid (Adam + bf16 write-back)"
        if kind == "update":
            return ("cm_update_kernel<true, true, true, false, false, false, false, 3, false> "
                    "(fused Adam + bf16 write-back + pack)")
        return f"cm_update_kernel ({kind}) (fused Adam + bf16 write-back + pack)"
    if deferred and kind == "update_handover":
        return ("rv_update_kernel Adam-only pass, then rv_update_kernel<true, false, false, false, "
                "false, false, true> (the interval's last step: Adam, then the sum of the "
                "interval's gradients into the hand-over)")
    if kind == "update_adam":
        return ("update_kernel (refresh steps) / rv_update_kernel (steps in place): Adam + bf16 "
                "write-back")
    return f"rv_update_kernel / update_kernel ({kind}) (fused Adam + bf16 write-back + pack)"


def traffic_settings(config: dict) -> str:
    """The settings of a run, beyond its workload and layout, that its
    launches' bytes depend on (from the `config` object of the bench line)."""
    keys = ("topk_ratio", "refresh_interval", "accum_interval", "zen_auto_tau",
            "zen_interval_decided_on", "offload", "first_step_stage", "packing")
    return json.dumps({k: config.get(k) for k in keys}, sort_keys=True)


def recorded_traffic(launch_kind: str, workload: str, variant: str, settings: str):
    """HBM bytes per launch of one launch kind, from rocprofv3 PMC counters
    (FETCH_SIZE and WRITE_SIZE runs, scaled by the reference copy stream's
    reading), if recorded for this workload, variant (layout, and for the
    eager path "-every-step"), run settings (`traffic_settings`) and the
    current kernel sources."""
    path = os.path.join(PROFILES, f"traffic_{workload}_{variant}.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    h = re.search(r"kernel_source_sha256_16:\s*([0-9a-f]+)", text)
    c = re.search(r"profiled_settings:\s*(\{.*\})", text)
    v = re.search(r"traffic_bytes_per_launch\[" + re.escape(launch_kind) +
                  r"\]:\s*([0-9.eE+]+)", text)
    if not h or not c or not v or h.group(1) != kernel_source_hash() or c.group(1) != settings:
        return None
    return float(v.group(1))


def calibrate_streams(dev, gib: float, reps: int = 10) -> dict:
    """The reference streams of zf_measure.h (the update pass's access
    pattern with no arithmetic) over `gib` GiB: read-only, copy and
    read-modify-write in place, each one untimed launch then `reps` timed
    ones (HIP events on the launch stream).  They are the process's first
    GPU work, so about 0.1 s of copies runs first: on a GPU that has just
    left idle the first milliseconds stream slower."""
    import torch
    import paper_2505_12242_amd as zf
    nb = int(gib * 2**30) // 16 * 16
    src = torch.empty(nb, dtype=torch.uint8, device=dev).fill_(1)
    dst = torch.empty(nb, dtype=torch.uint8, device=dev).fill_(2)
    sink = torch.zeros(1, dtype=torch.int32, device=dev)
    stream = torch.cuda.current_stream(dev)
    out = {"kernel": "stream_probe_kernel<0|1|2> (zf_stream_probe)", "GiB": gib}
    warm_ms, t_warm = 0.0, time.perf_counter()
    while warm_ms < 100.0 and time.perf_counter() - t_warm < 5.0:
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        zf.stream_probe(zf.PROBE_COPY, src, dst, nb, stream=stream)
        e1.record(stream)
        torch.cuda.synchronize(dev)
        warm_ms += e0.elapsed_time(e1)
    for kind, name, moved in ((zf.PROBE_READ, "read", nb), (zf.PROBE_COPY, "copy", 2 * nb),
                              (zf.PROBE_RMW, "rmw", 2 * nb)):
        args = ((src, sink) if kind == zf.PROBE_READ else (src, dst) if kind == zf.PROBE_COPY
                else (None, dst))
        zf.stream_probe(kind, *args, nb, key=0x9E3779B9, stream=stream)
        torch.cuda.synchronize(dev)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            zf.stream_probe(kind, *args, nb, key=0x9E3779B9, stream=stream)
        e1.record(stream)
        torch.cuda.synchronize(dev)
        ms = e0.elapsed_time(e1) / reps
        out[f"{name}_GB/s"] = round(moved / (ms * 1e-3) / 1e9, 1)
    del src, dst, sink
    torch.cuda.empty_cache()
    return out


UPDATE_NAMES = ("update", "update_first", "update_second", "update_handover", "update_adam",
                "update_adam_handover", "update_zen", "update_zen_first")


def default_packing(zen_tau, accum: int, refresh: int) -> str:
    """--packing's default: deferred, except Zen-auto with intervals longer
    than ZEN_DEFER_MAX steps (at most min(S, R)), which packs every step."""
    if zen_tau is not None and min(accum, refresh) > ZEN_DEFER_MAX:
        return "every-step"
    return "deferred"


def kernel_class(name: str):
    """Which entry of step_bytes a recorded launch belongs to."""
    if name in ("colnorm", "topk_select", "unpack"):
        return name
    if name == "handover_zen":
        return "unpack"
    if name in UPDATE_NAMES:
        return "update"
    return None


def main(argv=None) -> int:
    args = parse_args(argv)
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "bench.py measures the hot path on one GPU (one GPU's "
                                   "share of the work); --gpus must be 1"}), flush=True)
        return 2

    import torch
    import paper_2505_12242_amd as zf
    from workloads import get_workload

    if not torch.cuda.is_available():
        print(json.dumps({"error": "no GPU visible"}), flush=True)
        return 1
    dev = torch.device("cuda", 0)
    torch.cuda.set_device(dev)
    wl = get_workload(args.workload)
    over = {k: v for k, v in (("ratio", args.ratio), ("refresh", args.refresh),
                              ("accum", args.accum)) if v is not None}
    if over:
        wl = wl.with_(**over)
    if args.layers is not None:
        keep = tuple(mt for mt in wl.matrices if not mt.name.startswith("layers.")
                     or int(mt.name.split(".")[1]) < args.layers)
        wl = wl.with_(name=f"{wl.name}-first{args.layers}layers", matrices=keep)
    layout = zf.CHANNEL_MAJOR if args.layout == "channel-major" else zf.ROW_MAJOR
    hp = zf.AdamHparams(wl.hyper.lr, wl.hyper.beta1, wl.hyper.beta2, wl.hyper.eps,
                        wl.hyper.weight_decay)

    # reference streams first, while HBM is free
    calib = None
    if args.calibration_gib > 0:
        calib = calibrate_streams(dev, args.calibration_gib)
        print(f"# reference streams over {args.calibration_gib:g} GiB: read "
              f"{calib['read_GB/s']}, copy {calib['copy_GB/s']}, read-modify-write "
              f"{calib['rmw_GB/s']} GB/s", file=sys.stderr, flush=True)

    # Zen-auto: with deferred packing when decided on the device, channel-major,
    # and by default only for intervals of at most ZEN_DEFER_MAX steps (its
    # statistics re-read the interval's kept gradients at every step)
    packing = args.packing or default_packing(args.zen_tau, wl.accum, wl.refresh)
    deferred = (packing == "deferred" and not args.offload and not args.separate_handover
                and (args.zen_tau is None
                     or (not args.zen_on_host and args.layout == "channel-major")))
    if deferred:
        args.slots = max(args.slots, min(wl.accum, wl.refresh))
    t0 = time.perf_counter()
    shapes, ks, grad_slots, weights = build_set(wl, args.slots, dev, layout)
    sample = None
    one_thread_qs = []
    if not args.no_cpu_baseline:
        names = [mt.name for mt in wl.matrices]
        one_thread_qs = [q for q, nm in enumerate(names) if nm.startswith("layers.0.")] or [0]
        if args.cpu_sample == "layer":
            qs = one_thread_qs
        else:
            qs = list(range(len(shapes)))
        # the initial weights, before the GPU run updates them
        sample = HostSample(wl, qs, weights, layout)
    runner = zf.SelectiveUpdateRunner(shapes, wl.ratio, hp, wl.refresh, wl.accum, grad_slots,
                                      weights, device=dev, layout=layout, zen_tau=args.zen_tau,
                                      offload=args.offload, overlap=not args.no_overlap,
                                      host_threads=args.host_threads,
                                      fuse_handover=not args.separate_handover,
                                      refresh_pending=not args.refresh_waits,
                                      first_step_stage=not args.no_first_step_stage,
                                      zen_on_device=not args.zen_on_host,
                                      deferred_pack=deferred)
    fused = runner.keep_unpacked and runner.fuse_handover and args.zen_tau is None
    torch.cuda.synchronize()
    setup_s = time.perf_counter() - t0
    print(f"# setup {setup_s:.1f}s: {len(shapes)} matrices, {wl.params:,} params, "
          f"{torch.cuda.memory_allocated() / 2**30:.1f} GiB allocated", file=sys.stderr, flush=True)

    # stand-in model compute (offload mode): n_mm products of two 4096 x 4096
    # bf16 matrices, calibrated to model_compute_ms per step
    model = None
    if args.model_compute_ms > 0:
        if not args.offload:
            print(json.dumps({"error": "--model-compute-ms needs --offload"}))
            return 2
        ma = torch.randn(4096, 4096, device=dev, dtype=torch.bfloat16)
        mb = torch.randn(4096, 4096, device=dev, dtype=torch.bfloat16)
        mc = torch.empty_like(ma)
        for _ in range(3):
            torch.mm(ma, mb, out=mc)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(20):
            torch.mm(ma, mb, out=mc)
        e1.record()
        torch.cuda.synchronize()
        n_mm = max(1, round(args.model_compute_ms / (e0.elapsed_time(e1) / 20)))

        def model():
            for _ in range(n_mm):
                torch.mm(ma, mb, out=mc)

    for _ in range(args.warmup):
        if model is not None:
            model()
        runner.step()
    if args.offload:
        runner.sync()
        runner.stall_s = runner.host_update_s = 0.0
        th0 = runner.th
        pr0 = runner.pending_refreshes
    torch.cuda.synchronize()

    stream = torch.cuda.current_stream()
    spans = []  # (name, timed step index, start event, end event)
    cur = [0]

    @contextlib.contextmanager
    def recorder(name):
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record(stream)
        yield
        b.record(stream)
        spans.append((name, cur[0], a, b))

    kinds = []
    # the garbage collector stays off in the timed region: a collection there
    # is a host pause that a short step does not hide
    gc.collect()
    gc.disable()
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    for i in range(args.steps):
        cur[0] = i
        if model is not None:
            with recorder("model_compute"):
                model()
        kinds.append(runner.step(recorder=recorder))
    t_drain = time.perf_counter()
    if args.offload:
        runner.sync()  # the last deferred update lands inside the timed region
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    drain = time.perf_counter() - t_drain
    gc.enable()

    def model_bytes(kind, unfused=False):
        first, second = kind.step_in_interval == 1, kind.step_in_interval == 2
        if unfused:  # the unfused method: separate hand-over, fp32 first-step packing
            return step_bytes(shapes, ks, kind.refresh, first, kind.interval_end,
                              offload=args.offload)
        # (Zen-auto on the device: an end the caller forces is handed over
        # by the update itself)
        fh = fused or getattr(kind, "fused", False)
        return step_bytes(shapes, ks, kind.refresh, first, kind.interval_end,
                          offload=args.offload, fused_handover=fh, second=second,
                          stage=runner.use_stage, scored_handover=runner.score_handover,
                          deferred=runner.deferred, length=kind.step_in_interval,
                          zen=args.zen_tau is not None)

    def model_traffic(kind):
        first, second = kind.step_in_interval == 1, kind.step_in_interval == 2
        fh = fused or getattr(kind, "fused", False)
        return step_traffic(shapes, ks, kind.refresh, first, kind.interval_end,
                            offload=args.offload, fused_handover=fh, second=second,
                            stage=runner.use_stage, scored_handover=runner.score_handover,
                            deferred=runner.deferred, length=kind.step_in_interval,
                            zen=args.zen_tau is not None)

    build_total = sum(sum(model_bytes(k).values()) for k in kinds)
    unfused_total = sum(sum(model_bytes(k, True).values()) for k in kinds)
    value = build_total / wall / 1e9
    # what the reference streams predict for a pass that reads r and writes w
    # bytes: r / (read rate) + w / (write rate), the write rate inferred from
    # the copy stream (half reads, half writes)
    stream_rates = None
    if calib:
        rr = calib["read_GB/s"] * 1e9
        wr = 0.5 / (1.0 / (calib["copy_GB/s"] * 1e9) - 0.5 / rr)
        stream_rates = (rr, wr)
        calib["write_GB/s_inferred"] = round(wr / 1e9, 1)

    per = {}
    for name, i, a, b in spans:
        e = per.setdefault(name, {"ms": [], "bytes": 0, "unfused": 0, "rw": [0, 0]})
        e["ms"].append(a.elapsed_time(b))
        cls = kernel_class(name)
        if cls is not None:
            r, w = model_traffic(kinds[i])[cls]
            e["bytes"] += r + w
            e["rw"][0] += r
            e["rw"][1] += w
            e["unfused"] += model_bytes(kinds[i], True)[cls]
    kernels = {}
    for name, e in per.items():
        n = len(e["ms"])
        avg = sum(e["ms"]) / n
        k = {"launches": n, "avg_ms": round(avg, 4), "total_ms": round(sum(e["ms"]), 3)}
        if e["bytes"]:
            rate = e["bytes"] / n / (avg * 1e-3) / 1e9
            k.update({"GB_per_launch": round(e["bytes"] / n / 1e9, 3), "GB/s": round(rate, 1),
                      "frac_of_peak": round(rate / HBM_PEAK_GBS, 4)})
            if stream_rates:
                model_ms = (e["rw"][0] / stream_rates[0] + e["rw"][1] / stream_rates[1]) / n * 1e3
                k["read_fraction"] = round(e["rw"][0] / e["bytes"], 3)
                k["reference_stream_ms"] = round(model_ms, 4)
                k["frac_of_reference_stream"] = round(model_ms / avg, 4)
        kernels[name] = k

    # the dominant kernel: the fused Adam + pack pass in its middle-step form
    # (states in place, accumulation; no hand-over): its bytes per launch are
    # the unfused method's per-unit figures, 28 per selected and 10 per unselected
    # element; else the launch kind with the most time
    timed = [nm for nm in per if per[nm]["bytes"]]
    dom = "update" if "update" in per else (max(timed, key=lambda nm: sum(per[nm]["ms"]))
                                            if timed else None)
    roof = None
    if dom is not None:
        e = per[dom]
        n = len(e["ms"])
        avg = sum(e["ms"]) / n
        nbytes = (e["unfused"] if dom == "update" else e["bytes"]) / n
        achieved = nbytes / (avg * 1e-3) / 1e9
        kname = launch_kernels(dom, layout == zf.CHANNEL_MAJOR, runner.deferred,
                               runner.use_stage, bool(runner.score_handover))
        roof = {
            "kernel": kname,
            "launch_kind": dom,
            "bound": "hbm",
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": None,
            "bytes_per_launch": round(nbytes),
            "byte_model": "unfused per-unit figures" if dom == "update" else "build",
            "avg_launch_ms": round(avg, 4),
            "frac_of_reference_stream": kernels[dom].get("frac_of_reference_stream"),
        }

    result = {
        "metric": "GB/s and fraction of HBM peak per full step; params/s",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall / args.steps * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp32",
        "data": "synthetic",
        "frac_of_hbm_peak": round(value / HBM_PEAK_GBS, 4),
        "params_per_s": round(wl.params * args.steps / wall, 1),
        "config": {
            "workload": wl.name,
            "matrices": len(shapes),
            "params": wl.params,
            "layout": args.layout,
            "grad_dtype": "bf16",
            "state_dtype": "fp32",
            "topk_ratio": wl.ratio,
            "refresh_interval": wl.refresh,
            "accum_interval": wl.accum,
            "zen_auto_tau": args.zen_tau,
            "zen_interval_decided_on": (None if args.zen_tau is None else
                                        "device" if runner.zen_device else "host"),
            "offload": args.offload,
            "model_compute_ms": args.model_compute_ms or None,
            "interval_ends": sum(1 for k in kinds if k.interval_end),
            "first_step_stage": runner.use_stage,
            "packing": ("deferred: the kept gradients summed again at every step for the "
                        "Zen-auto statistics" if runner.deferred and args.zen_tau is not None
                        else "deferred to the interval's last step" if runner.deferred else
                        "every step"),
            "handover": ("written by the score pass (one-step intervals)"
                         if runner.score_handover and wl.refresh == 1 else
                         "fused into the interval's last update") if fused else
                        ("device -> host copy of the packed buffer" if args.offload
                         else "fused into the update at forced ends, else the gated pass"
                         if runner.zen_device else "separate unpack pass"),
            "grad_slots": args.slots,
        },
        "byte_models": {
            "build": {"GB_per_step": round(build_total / args.steps / 1e9, 3),
                      "GB/s": round(value, 1), "frac_of_peak": round(value / HBM_PEAK_GBS, 4),
                      "what": "bytes this build's kernels move (value)"},
            "unfused": {"GB_per_step": round(unfused_total / args.steps / 1e9, 3),
                        "GB/s": round(unfused_total / wall / 1e9, 1),
                        "frac_of_peak": round(unfused_total / wall / 1e9 / HBM_PEAK_GBS, 4),
                        "what": "the unfused method's bytes: packing every step in fp32, a "
                                "separate hand-over pass"},
        },
        "kernels": kernels,
        "reference_streams": calib,
        "roofline": roof,
    }
    if roof is not None:
        roof["traffic"] = recorded_traffic(dom, wl.name, args.layout + (
            "" if runner.deferred else "-every-step"), traffic_settings(result["config"]))
    if args.offload:
        # host side of the deferred update: per unselected element it reads
        # the accumulated sum (4 B), reads and writes p, m, v (24 B) and
        # writes the bf16 weight (2 B); the device -> host copy moves 4 B
        intervals = runner.th - th0
        unsel = sum(n * (m - k) for (n, m), k in zip(shapes, ks))
        host_bytes = 30 * unsel * intervals
        result["offload"] = {
            "overlap": not args.no_overlap,
            "pending_refreshes": runner.pending_refreshes - pr0,
            "host_threads": runner.host_threads,
            "intervals": intervals,
            "host_update_s": round(runner.host_update_s, 4),
            "host_update_GB/s": round(host_bytes / runner.host_update_s / 1e9, 2)
            if runner.host_update_s else None,
            "host_params_per_s": round(unsel * intervals / runner.host_update_s, 1)
            if runner.host_update_s else None,
            "d2h_GB_per_interval": round(4 * unsel / 1e9, 3),
            "stall_s": round(runner.stall_s, 4),
            "stall_ms_per_step": round(runner.stall_s / args.steps * 1e3, 3),
            "store": "pinned host memory, read in place by the swap kernels",
            # GPU time of the recorded launches (hot path, write-back and the
            # stand-in model compute) against the wall time: what is left is
            # the GPU waiting for the host side
            "model_compute_ms_per_step": round(
                sum(per.get("model_compute", {"ms": []})["ms"]) / args.steps, 3),
            "gpu_busy_ms_per_step": round(
                sum(sum(v["ms"]) for v in per.values()) / args.steps, 3),
            "gpu_idle_ms_per_step": round(
                wall / args.steps * 1e3 - sum(sum(v["ms"]) for v in per.values()) / args.steps,
                3),
            # the last interval's copy, host update and write-back finish after
            # the last step (the drain): the idle time without it is what a
            # longer run approaches
            "drain_s": round(drain, 4),
            "gpu_idle_ms_per_step_without_drain": round(
                (wall - drain) / args.steps * 1e3
                - sum(sum(v["ms"]) for v in per.values()) / args.steps, 3),
        }
    runner.close()
    if sample is not None:
        try:
            print("# timing the CPU oracle on a sample ...", file=sys.stderr, flush=True)
            sample.add_grads(grad_slots, args.cpu_sample_steps)
            del grad_slots, weights
            torch.cuda.empty_cache()
            info = host_info()
            workers = min(16, info["nproc"])
            cb = cpu_baseline(wl, shapes, ks, sample, one_thread_qs, workers)
            best = cb.get("all_cores") or dict(cb["one_thread"], processes=1)
            result["cpu_baseline"] = {
                "value": best["GB/s"],
                "unit": "GB/s",
                "params_per_s": best["params_per_s"],
                "cores": best["processes"],
                "kind": "oracle",
                "sample": (best["sample"] + f" of the R={wl.refresh}, S={wl.accum} schedule, "
                           f"numpy oracle, one process per core"),
                "one_thread": cb["one_thread"],
                "all_cores": best,
                "host": info,
            }
        finally:
            sample.close()
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
