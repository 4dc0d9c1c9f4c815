"""The bench's byte model (the algorithmic bytes that GB/s and the roofline
fraction are computed from), checked on the CPU against hand counts:

* per parameter at 10% on the 4096 x 4096 matrix: refresh + first step
  2 + 8.2 B, a middle step 11.8 B, an interval end with the fused hand-over
  10 + 2.8 + 0.4 B;
* the bf16 first-step stage: refresh + first step 4 + 2.8 B (the score pass
  writes every channel's stage row, the update runs Adam alone), a plain
  first step 2.8 + 3.6 B, the second step 2.8 + 7.2 B; a refresh step that
  is a whole interval 6 + 3.2 B (the score pass writes the hand-over);
* the 16-step R = S = 4 schedule of the 7B set: 89.63 GB per step with a
  separate hand-over pass, 77.50 GB fused, 68.75 GB with the stage.
"""
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

bench = pytest.importorskip("bench")
from workloads.configs import get_workload, shapes as wl_shapes  # noqa: E402

N = M = 4096
K = 410  # round(0.1 * 4096)
U = M - K


def per_param(**kw):
    b = bench.step_bytes([(N, M)], [K], **kw)
    return sum(b.values()) / (N * M)


def test_single_matrix_step_types():
    refresh_first = per_param(refresh=True, first=True, end=False)
    want = (2 * N * M + 4 * M + 8 * M + 12 * (M // 64) + 28 * N * K + 6 * N * U) / (N * M)
    assert refresh_first == pytest.approx(want, rel=1e-12)
    assert per_param(refresh=False, first=False, end=False) == pytest.approx(
        (28 * N * K + 10 * N * U) / (N * M), rel=1e-12)
    assert per_param(refresh=False, first=False, end=True, fused_handover=True) == pytest.approx(
        (28 * N * K + 10 * N * U + 4 * N * K) / (N * M), rel=1e-12)
    # with the stage
    staged = per_param(refresh=True, first=True, end=False, stage=True, fused_handover=True)
    assert staged == pytest.approx(
        (4 * N * M + 4 * M + 8 * M + 12 * (M // 64) + 28 * N * K) / (N * M), rel=1e-12)
    assert per_param(refresh=False, first=True, end=False, stage=True) == pytest.approx(
        (28 * N * K + 4 * N * U) / (N * M), rel=1e-12)
    assert per_param(refresh=False, first=False, end=False, second=True, stage=True) == \
        pytest.approx((28 * N * K + 8 * N * U) / (N * M), rel=1e-12)
    # the stage with a separate hand-over pass (Zen-auto): the refresh packs
    # into the stage in the update, a one-step interval's pass reads it
    assert per_param(refresh=True, first=True, end=False, stage=True) == pytest.approx(
        (2 * N * M + 4 * M + 8 * M + 12 * (M // 64) + 28 * N * K + 4 * N * U) / (N * M),
        rel=1e-12)
    assert per_param(refresh=False, first=True, end=True, stage=True) == pytest.approx(
        (28 * N * K + 4 * N * U + 2 * N * U + 4 * N * M) / (N * M), rel=1e-12)
    # a refresh step that is a one-step interval: hand-over from the score pass
    assert per_param(refresh=True, first=True, end=True, fused_handover=True) == pytest.approx(
        (2 * N * M + 4 * M + 8 * M + 12 * (M // 64) + 28 * N * K + 6 * N * U + 4 * N * K)
        / (N * M), rel=1e-12)
    assert per_param(refresh=True, first=True, end=True, fused_handover=True, stage=True) == \
        pytest.approx((6 * N * M + 4 * M + 8 * M + 12 * (M // 64) + 28 * N * K + 4 * N * K)
                      / (N * M), rel=1e-12)


def test_7b_schedule_totals():
    wl = get_workload("llama2-7b-full")
    shp = wl_shapes(wl.matrices)
    ks = [int(r) for r in (bench_k(m, wl.ratio) for _, m in shp)]
    from paper_2505_12242_amd.runner import schedule

    def avg(**kw):
        tot = 0
        for t in range(1, 17):
            kd = schedule(t, 4, 4)
            tot += sum(bench.step_bytes(shp, ks, kd.refresh, kd.step_in_interval == 1,
                                        kd.interval_end, second=kd.step_in_interval == 2,
                                        **kw).values())
        return tot / 16 / 1e9

    assert avg() == pytest.approx(89.63, abs=0.01)
    assert avg(fused_handover=True) == pytest.approx(77.50, abs=0.01)
    assert avg(fused_handover=True, stage=True) == pytest.approx(68.75, abs=0.01)


def bench_k(m, ratio):
    import math
    return min(m, max(0, math.floor(ratio * m + 0.5)))


def test_read_write_split():
    """step_traffic splits each kernel's bytes into reads and writes; their
    sums are step_bytes.  A middle step of the fused update reads G and the
    selected states (2 + 12 B) and the previous sums (4 B), and writes the
    states and the weight (12 + 2 B) and the new sums (4 B)."""
    shapes, ks = [(64, 100), (7, 33)], [10, 3]
    for args in [(True, True, False), (False, False, False), (False, False, True),
                 (True, True, True)]:
        for kw in ({}, {"fused_handover": True, "stage": True}, {"offload": True},
                   {"fused_handover": True, "stage": True, "second": True}):
            t = bench.step_traffic(shapes, ks, *args, **kw)
            b = bench.step_bytes(shapes, ks, *args, **kw)
            assert {c: r + w for c, (r, w) in t.items()} == b
    t = bench.step_traffic(shapes, ks, False, False, False)
    nk = 64 * 10 + 7 * 3
    nu = 64 * 90 + 7 * 30
    assert t["update"] == [14 * nk + 6 * nu, 14 * nk + 4 * nu]


def test_deferred_packing_bytes():
    """Deferred packing: steps before an interval's last move the selected
    part only (28 B per selected element); the last step of L steps reads
    each step's gradient once at the unselected elements (2 B each) and
    writes the hand-over (4 B per element, zeros at the selected)."""
    n, m, k = 4096, 4096, 410
    u = m - k
    sh, ks = [(n, m)], [k]
    kw = dict(fused_handover=True, deferred=True)
    assert bench.step_bytes(sh, ks, True, True, False, length=1, **kw) == {
        "colnorm": 2 * n * m + 4 * m, "topk_select": 8 * m + 12 * 64, "update": 28 * n * k,
        "unpack": 0}
    assert bench.step_bytes(sh, ks, False, False, False, length=3, **kw)["update"] == 28 * n * k
    for L in (2, 4, 8):
        assert bench.step_bytes(sh, ks, False, False, True, length=L, **kw)["update"] == \
            28 * n * k + 4 * n * k + (2 * L + 4) * n * u
    # a refresh step that is a whole interval hands over from the score pass
    b = bench.step_bytes(sh, ks, True, True, True, length=1, **kw)
    assert b["colnorm"] == 6 * n * m + 4 * m and b["update"] == 32 * n * k


def test_zen_deferred_packing_bytes():
    """Zen-auto with deferred packing: a step at position p of its interval
    reads the kept gradients at the unselected elements (2p B each) for the
    statistics and writes nothing for them; an end the caller forces writes
    the hand-over from the update (4 B per element, zeros at the selected),
    any other end from the gated pass, which reads the p gradients again.
    Over an interval of 4 steps ended by force that is 24 B per unselected
    element, against 32 when packing every step with the stage."""
    n, m, k = 4096, 4096, 410
    u = m - k
    sh, ks = [(n, m)], [k]
    kw = dict(deferred=True, zen=True)
    b = bench.step_bytes(sh, ks, True, True, False, length=1, **kw)
    assert b == {"colnorm": 2 * n * m + 4 * m, "topk_select": 8 * m + 12 * 64,
                 "update": 28 * n * k + 2 * n * u, "unpack": 0}
    for p in (2, 3, 6):
        assert bench.step_bytes(sh, ks, False, False, False, length=p, **kw)["update"] == \
            28 * n * k + 2 * p * n * u
        forced = bench.step_bytes(sh, ks, False, False, True, length=p, fused_handover=True, **kw)
        assert forced["update"] == 28 * n * k + 4 * n * k + (2 * p + 4) * n * u
        assert forced["unpack"] == 0
        trig = bench.step_bytes(sh, ks, False, False, True, length=p, **kw)
        assert trig["update"] == 28 * n * k + 2 * p * n * u
        assert trig["unpack"] == 2 * p * n * u + 4 * n * m
    per_u = sum(bench.step_bytes([(1, 1000)], [0], False, p == 1, p == 4, length=p,
                                 fused_handover=p == 4, **kw)["update"] for p in (1, 2, 3, 4))
    assert per_u == 24 * 1000


def test_recorded_traffic_needs_the_profiled_settings(tmp_path, monkeypatch):
    """PMC traffic recorded under profiles/ applies to a bench line only for
    the same kernel sources, workload, layout variant and run settings (ratio,
    schedule, packing, Zen-auto, offload): a run at another ratio or refresh
    interval moves other bytes and reports no traffic."""
    cfg = {"topk_ratio": 0.1, "refresh_interval": 4, "accum_interval": 4, "zen_auto_tau": None,
           "zen_interval_decided_on": None, "offload": False, "first_step_stage": False,
           "packing": "deferred to the interval's last step", "grad_slots": 4}
    text = ("Machine-readable:\n\n"
            f"kernel_source_sha256_16: {bench.kernel_source_hash()}\n"
            f"profiled_settings: {bench.traffic_settings(cfg)}\n"
            "traffic_bytes_per_launch[update_handover]: 9.4e+10\n")
    (tmp_path / "traffic_wl_channel-major.md").write_text(text)
    monkeypatch.setattr(bench, "PROFILES", str(tmp_path))
    get = bench.recorded_traffic
    assert get("update_handover", "wl", "channel-major", bench.traffic_settings(cfg)) == 9.4e10
    # settings outside the byte model (the ring's slot count) do not matter
    assert get("update_handover", "wl", "channel-major",
               bench.traffic_settings(dict(cfg, grad_slots=3))) == 9.4e10
    for change in ({"topk_ratio": 0.25}, {"refresh_interval": 1}, {"zen_auto_tau": 1.0},
                   {"packing": "every step"}, {"offload": True}):
        assert get("update_handover", "wl", "channel-major",
                   bench.traffic_settings(dict(cfg, **change))) is None, change
    assert get("update_adam", "wl", "channel-major", bench.traffic_settings(cfg)) is None
    assert get("update_handover", "wl", "row-major", bench.traffic_settings(cfg)) is None
    (tmp_path / "traffic_wl_channel-major.md").write_text(
        text.replace(bench.kernel_source_hash(), "0" * 16))
    assert get("update_handover", "wl", "channel-major", bench.traffic_settings(cfg)) is None


def test_committed_profiles_record_their_settings():
    """Every committed traffic summary names the settings it was taken with,
    and the default 7B line's settings match the headline profile."""
    import glob
    import json
    paths = glob.glob(os.path.join(ROOT, "profiles", "traffic_*.md"))
    assert paths
    for path in paths:
        text = open(path).read()
        line = [ln for ln in text.splitlines() if ln.startswith("profiled_settings:")]
        assert len(line) == 1, path
        json.loads(line[0].split(":", 1)[1])
    head = open(os.path.join(ROOT, "profiles", "traffic_llama2-7b-full_channel-major.md")).read()
    assert '"refresh_interval": 4' in head and '"topk_ratio": 0.1' in head


def test_default_packing():
    """Deferred packing by default; Zen-auto keeps it for intervals of at most
    ZEN_DEFER_MAX steps, where its per-step re-reads, p(p + 1) + 4 bytes per
    unselected element over p >= 2 steps, stay below packing's 10p - 8 (the
    bytes cross over at 8 steps; the time measured earlier, its read-heavy
    passes streaming slower)."""
    assert bench.ZEN_DEFER_MAX == 6
    assert bench.default_packing(None, 8, 8) == "deferred"
    assert bench.default_packing(None, 16, 16) == "deferred"
    assert bench.default_packing(1.0, 4, 4) == "deferred"
    assert bench.default_packing(1.0, 6, 16) == "deferred"
    assert bench.default_packing(1.0, 8, 8) == "every-step"
    assert bench.default_packing(0.5, 16, 7) == "every-step"
    for p in range(2, bench.ZEN_DEFER_MAX + 1):
        assert p * (p + 1) + 4 < 10 * p - 8, p
    assert 8 * 9 + 4 > 10 * 8 - 8
