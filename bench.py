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
KERNEL_SOURCES = [os.path.join(ROOT, "paper_2505_12242_amd", "csrc", f)
                  for f in ("zf_device.hpp", "zf_internal.hpp", "zf_kernels.hip",
                            "zf_kernels_cm.hip", "zf_kernels_rv.hip")]


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
    ap.add_argument("--ratio", type=float, default=None, help="override the top-k ratio")
    ap.add_argument("--refresh", type=int, default=None, help="override the refresh interval R")
    ap.add_argument("--accum", type=int, default=None, help="override the accumulation interval S")
    ap.add_argument("--zen-tau", type=float, default=None,
                    help="run Zen-auto (adaptive interval, at most --accum steps) with this "
                         "threshold instead of the fixed schedule")
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
    ap.add_argument("--separate-handover", action="store_true",
                    help="hand over with a separate unpack pass after the last update of an "
                         "interval instead of fusing it into that update")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-sample-steps", type=int, default=4)
    ap.add_argument("--calibration-copy-gib", type=float, default=1.0,
                    help="size of the plain copy launched once for PMC calibration (0: skip)")
    return ap.parse_args(argv)


# ---------------------------------------------------------------------------
# byte model: the bytes each kernel must move, per matrix
# ---------------------------------------------------------------------------

def step_bytes(shapes, ks, refresh: bool, first: bool, end: bool, offload: bool = False,
               fused_handover: bool = False, second: bool = False, stage: bool = False,
               scored_handover: bool = None) -> dict:
    """Algorithmic HBM bytes of one step, by kernel.

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
    """
    if scored_handover is None:
        scored_handover = stage
    out = {"colnorm": 0, "topk_select": 0, "update": 0, "unpack": 0}
    for (n, m), k in zip(shapes, ks):
        u = m - k
        staged_refresh = refresh and stage and fused_handover and not end
        scored_end = refresh and stage and scored_handover and fused_handover and end and first
        if refresh:
            out["colnorm"] += (2 * n * m + 4 * m + (2 * n * m if staged_refresh else 0)
                               + (4 * n * m if scored_end else 0))
            out["topk_select"] += 8 * m + 12 * ((m + 63) // 64)
        if staged_refresh or scored_end:
            per_u = 0
        elif first:
            # the fused hand-over of a one-step interval writes no packed values
            per_u = 4 if (stage and not (end and fused_handover)) else 6
        else:
            per_u = 8 if (stage and second) else 10
        out["update"] += 28 * n * k + per_u * n * u
        if end:
            if offload:
                out["unpack"] += 4 * n * u + 2 * n * u
            elif fused_handover:
                out["update"] += 4 * n * k
            else:
                # the separate pass reads the stage after a one-step interval
                out["unpack"] += (2 if (stage and first) else 4) * n * u + 4 * n * m
    return out


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

def cpu_baseline(wl, shapes, ks, grad_slots, weights0, steps: int, layout: int = 0) -> dict:
    """Times the oracle (as it stands) over the first decoder layer's seven
    matrices for `steps` steps of the workload's schedule, on the host.
    Inputs are copied to the host in the logical [out, in] layout before
    timing."""
    import numpy as np
    import torch
    import oracle as O

    def logical(t):
        return t if layout == 0 else t.t()

    qs = [q for q, mt in enumerate(wl.matrices) if mt.name.startswith("layers.0.")]
    if not qs:
        qs = [0]
    hp = wl.hyper
    host_g = {}
    for q in qs:
        for t in range(1, steps + 1):
            s = (t - 1) % len(grad_slots)
            if (q, s) not in host_g:
                host_g[(q, s)] = np.ascontiguousarray(
                    logical(grad_slots[s][q]).contiguous().view(torch.int16).cpu().numpy()
                    .view(np.uint16))
    elapsed = 0.0
    nbytes = 0
    for q in qs:
        W = weights0[q]
        orc = O.MatrixOracle(O.widen(W), W, wl.ratio, hp.lr, hp.beta1, hp.beta2, hp.eps,
                             hp.weight_decay, wl.refresh, wl.accum)
        for t in range(1, steps + 1):
            G = host_g[(q, (t - 1) % len(grad_slots))]
            t0 = time.perf_counter()
            out = orc.step(G)
            elapsed += time.perf_counter() - t0
            kind = out["kind"]
            b = step_bytes([shapes[q]], [ks[q]], kind.refresh, kind.step_in_interval == 1,
                           kind.interval_end)
            nbytes += sum(b.values())
    params = sum(shapes[q][0] * shapes[q][1] for q in qs)
    return {
        "value": round(nbytes / elapsed / 1e9, 4),
        "unit": "GB/s",
        "params_per_s": round(params * steps / elapsed, 1),
        "seconds": round(elapsed, 3),
        "cores": 1,
        "kind": "oracle",
        "sample": (f"{len(qs)} matrices of the first decoder layer "
                   f"({params:,} params), steps 1-{steps} of the R={wl.refresh}, "
                   f"S={wl.accum} schedule, numpy oracle on one host thread"),
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


def recorded_traffic(kernel: str, workload: str):
    """Bytes per launch of the fused update kernel measured with rocprofv3
    PMC counters (scaled by a plain streaming kernel's counter reading), if
    recorded for this workload and the current kernel source."""
    path = os.path.join(PROFILES, f"{kernel}_{workload}_traffic.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    h = re.search(r"kernel_source_sha256_16:\s*([0-9a-f]+)", text)
    v = re.search(r"traffic_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not h or not v or h.group(1) != kernel_source_hash():
        return None
    return float(v.group(1))


# ---------------------------------------------------------------------------

def main(argv=None) -> int:
    args = parse_args(argv)
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(json.dumps({"error": "bench.py measures the hot path on one GPU (one GPU's "
                                   "share of the work); --gpus must be 1"}), flush=True)
        return 2

    import numpy as np
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
    layout = zf.CHANNEL_MAJOR if args.layout == "channel-major" else zf.ROW_MAJOR
    hp = zf.AdamHparams(wl.hyper.lr, wl.hyper.beta1, wl.hyper.beta2, wl.hyper.eps,
                        wl.hyper.weight_decay)

    t0 = time.perf_counter()
    shapes, ks, grad_slots, weights = build_set(wl, args.slots, dev, layout)
    weights0 = None
    if not args.no_cpu_baseline:
        qs0 = [q for q, mt in enumerate(wl.matrices) if mt.name.startswith("layers.0.")] or [0]
        weights0 = {}
        for q in qs0:
            w = weights[q] if layout == zf.ROW_MAJOR else weights[q].t()
            weights0[q] = w.contiguous().view(torch.int16).cpu().numpy().view(np.uint16)
    runner = zf.SelectiveUpdateRunner(shapes, wl.ratio, hp, wl.refresh, wl.accum, grad_slots,
                                      weights, device=dev, layout=layout, zen_tau=args.zen_tau,
                                      offload=args.offload, overlap=not args.no_overlap,
                                      host_threads=args.host_threads,
                                      fuse_handover=not args.separate_handover,
                                      refresh_pending=not args.refresh_waits,
                                      first_step_stage=not args.no_first_step_stage)
    fused = runner.keep_unpacked and runner.fuse_handover and args.zen_tau is None
    torch.cuda.synchronize()
    setup_s = time.perf_counter() - t0
    print(f"# setup {setup_s:.1f}s: {len(shapes)} matrices, {wl.params:,} params, "
          f"{torch.cuda.memory_allocated() / 2**30:.1f} GiB allocated", file=sys.stderr, flush=True)

    # one plain streaming kernel of known size (reads and writes exactly
    # calibration_copy_gib GiB each): the calibration point for PMC counters
    # (then timed over three more launches: a plain read+write stream on
    # this box, reported beside the roofline as context)
    stream_ref = None
    if args.calibration_copy_gib > 0:
        nb = int(args.calibration_copy_gib * 2**30)
        src = torch.empty(nb // 4, dtype=torch.float32, device=dev).fill_(4.0)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        torch.sqrt(src, out=dst)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(3):
            torch.sqrt(src, out=dst)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / 3
        stream_ref = {"kernel": f"torch.sqrt over {args.calibration_copy_gib:g} GiB fp32 "
                                "(reads and writes that much)",
                      "GB/s": round(2 * nb / (ms * 1e-3) / 1e9, 1)}
        del src, dst

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
    spans = []  # (name, start event, end event)

    @contextlib.contextmanager
    def recorder(name):
        a = torch.cuda.Event(enable_timing=True)
        b = torch.cuda.Event(enable_timing=True)
        a.record(stream)
        yield
        b.record(stream)
        spans.append((name, a, b))

    kinds = []
    # the garbage collector stays off in the timed region: a collection there
    # is a host pause that a short step does not hide
    gc.collect()
    gc.disable()
    torch.cuda.synchronize()
    w0 = time.perf_counter()
    for _ in range(args.steps):
        if model is not None:
            with recorder("model_compute"):
                model()
        kinds.append(runner.step(recorder=recorder))
    if args.offload:
        runner.sync()  # the last deferred update lands inside the timed region
    torch.cuda.synchronize()
    wall = time.perf_counter() - w0
    gc.enable()

    per_kernel_ms = {}
    for name, a, b in spans:
        per_kernel_ms.setdefault(name, []).append(a.elapsed_time(b))
    totals = {"colnorm": 0, "topk_select": 0, "update": 0, "unpack": 0}
    for kind in kinds:
        b = step_bytes(shapes, ks, kind.refresh, kind.step_in_interval == 1, kind.interval_end,
                       offload=args.offload, fused_handover=fused,
                       second=kind.step_in_interval == 2, stage=runner.use_stage,
                       scored_handover=runner.score_handover)
        for key in totals:
            totals[key] += b[key]
    all_bytes = sum(totals.values())
    update_bytes = totals["update"]  # both update kinds
    upd_ms = [ms for name, lst in per_kernel_ms.items() if name.startswith("update")
              for ms in lst]
    upd_launches = len(upd_ms)
    upd_avg_ms = sum(upd_ms) / max(upd_launches, 1)
    achieved = update_bytes / upd_launches / (upd_avg_ms * 1e-3) / 1e9 if upd_launches else 0.0

    value = all_bytes / wall / 1e9
    kernels = {}
    for name, lst in per_kernel_ms.items():
        kernels[name] = {"launches": len(lst), "avg_ms": round(sum(lst) / len(lst), 4)}
    for name in ("colnorm", "topk_select", "unpack"):
        if name in per_kernel_ms and totals[name]:
            tot_ms = sum(per_kernel_ms[name])
            kernels[name]["GB/s"] = round(totals[name] / (tot_ms * 1e-3) / 1e9, 1)

    upd_kernel = "cm_update_kernel" if layout == zf.CHANNEL_MAJOR else "update_kernel"
    if args.zen_tau is not None:
        upd_kernel += " (with Zen-auto statistics)"
    traffic = recorded_traffic(upd_kernel, wl.name)
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
            "offload": args.offload,
            "model_compute_ms": args.model_compute_ms or None,
            "interval_ends": sum(1 for k in kinds if k.interval_end),
            "first_step_stage": runner.use_stage,
            "handover": "fused into the interval's last update" if fused else
                        ("device -> host copy of the packed buffer" if args.offload
                         else "separate unpack pass"),
            "grad_slots": args.slots,
            "algorithmic_GB_per_step": round(all_bytes / args.steps / 1e9, 3),
        },
        "kernels": kernels,
        "roofline": {
            "kernel": (upd_kernel if layout == zf.CHANNEL_MAJOR else
                       "rv_update_kernel (steps in place, hand-over) and update_kernel "
                       "(refresh steps)") + " (fused Adam + bf16 write-back + pack)",
            "bound": "hbm",
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBS, 4),
            "traffic": traffic,
            "bytes_per_launch": round(update_bytes / max(upd_launches, 1)),
            "avg_launch_ms": round(upd_avg_ms, 4),
            "stream_reference": (dict(stream_ref, update_frac_of_it=round(
                achieved / stream_ref["GB/s"], 4)) if stream_ref else None),
        },
    }
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
                sum(per_kernel_ms.get("model_compute", [])) / args.steps, 3),
            "gpu_busy_ms_per_step": round(
                sum(sum(v) for v in per_kernel_ms.values()) / args.steps, 3),
            "gpu_idle_ms_per_step": round(
                wall / args.steps * 1e3 - sum(sum(v) for v in per_kernel_ms.values()) / args.steps,
                3),
        }
    if not args.no_cpu_baseline:
        print("# timing the CPU oracle on a sample ...", file=sys.stderr, flush=True)
        result["cpu_baseline"] = cpu_baseline(wl, shapes, ks, grad_slots, weights0,
                                              args.cpu_sample_steps, layout)
    runner.close()
    print(json.dumps(result), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
