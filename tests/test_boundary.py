"""The C ABI without a GPU: the library loads, exports every function that
include/zf.h declares, and rejects invalid arguments on the host before any
HIP call (fake device addresses are never dereferenced)."""
import ctypes
import math
import os
import re

import pytest

from tests.conftest import ROOT

zf = pytest.importorskip("paper_2505_12242_amd")
from paper_2505_12242_amd import _lib  # noqa: E402

LIB = _lib.LIB
OK, EINVAL, EWS = _lib.ZF_OK, _lib.ZF_EINVAL, _lib.ZF_EWORKSPACE
RM, CM = _lib.ROW_MAJOR, _lib.CHANNEL_MAJOR
A = 0x7F0000000000  # a 256-byte aligned fake device address
B = A + (1 << 30)
C = A + (2 << 30)
D = A + (3 << 30)
E = A + (4 << 30)


def header_functions():
    """Every function declared in include/*.h."""
    names = set()
    inc = os.path.join(ROOT, "include")
    for h in sorted(os.listdir(inc)):
        if h.endswith(".h"):
            text = re.sub(r"/\*.*?\*/", "", open(os.path.join(inc, h)).read(), flags=re.S)
            names |= set(re.findall(r"\b(zf_[a-z0-9_]+)\s*\(", text))
    return sorted(names)


def test_every_declared_function_is_exported_and_bound():
    names = header_functions()
    assert len(names) >= 16
    raw = ctypes.CDLL(_lib.LIB_PATH)
    bound = {s[0] for s in _lib.SIGNATURES}
    for name in names:
        assert hasattr(raw, name), name
        assert name in bound, name


def test_status_strings():
    for s in range(5):
        assert LIB.zf_status_string(s).decode().startswith("ZF_")
    assert b"unknown" in LIB.zf_status_string(99)
    assert LIB.zf_last_hip_error() == 0


@pytest.mark.parametrize("ratio,m,k", [(0.1, 4096, 410), (0.25, 2, 1), (0.0, 5, 0), (1.0, 5, 5),
                                       (0.05, 11008, 550), (0.1, 28672, 2867), (0.5, 0, 0)])
def test_k_from_ratio(ratio, m, k):
    assert LIB.zf_k_from_ratio(ratio, m) == k


@pytest.mark.parametrize("ratio,m", [(-0.01, 5), (1.01, 5), (math.nan, 5), (0.5, -1)])
def test_k_from_ratio_invalid(ratio, m):
    assert LIB.zf_k_from_ratio(ratio, m) == -1


def sel(m, k, base=C):
    words = (m + 63) // 64
    return _lib.ZfSelection(base, base + 4 * max(k, 1) + 256, base + (1 << 20), base + (2 << 20))


def test_colnorm_validation():
    ws = LIB.zf_colnorm_workspace_bytes(64, 64, RM)
    assert ws > 0 and LIB.zf_colnorm_workspace_bytes(0, 64, RM) == 0
    assert LIB.zf_colnorm_workspace_bytes(64, 64, CM) == 0
    call = LIB.zf_colnorm
    assert call(None, 4, 4, 4, RM, B, C, ws, None) == EINVAL          # null gradient
    assert call(A, 4, 4, 3, RM, B, C, ws, None) == EINVAL             # ld < m
    assert call(A, 4, 4, 4, 7, B, C, ws, None) == EINVAL              # unknown layout
    assert call(A + 1, 4, 4, 4, RM, B, C, ws, None) == EINVAL         # misaligned bf16
    assert call(A, 4, 4, 4, RM, B + 2, C, ws, None) == EINVAL         # misaligned fp32
    assert call(A, -1, 4, 4, RM, B, C, ws, None) == EINVAL            # n < 0
    assert call(A, 4, 4, 4, RM, A + 8, C, ws, None) == EINVAL         # output inside gradient
    assert call(A, 64, 64, 64, RM, B, None, 0, None) == EWS           # no workspace
    assert call(A, 64, 64, 64, RM, B, C, ws - 8, None) == EWS         # small workspace
    assert call(A, 4, 0, 4, RM, None, None, 0, None) == OK            # m = 0: nothing to do
    # channel-major: the gradient is [m][ld >= n]
    assert call(A, 8, 4, 7, CM, B, None, 0, None) == EINVAL           # ld < n
    assert call(A, 8, 0, 8, CM, None, None, 0, None) == OK


def test_topk_validation():
    s = sel(100, 10)
    call = LIB.zf_topk_select
    kout = ctypes.c_int64(-7)
    assert call(A, 100, 1.5, ctypes.byref(s), ctypes.byref(kout), None) == EINVAL
    assert call(A, 100, math.nan, ctypes.byref(s), None, None) == EINVAL
    assert call(A, 100, 0.1, None, None, None) == EINVAL
    assert call(None, 100, 0.1, ctypes.byref(s), None, None) == EINVAL
    bad = _lib.ZfSelection(C, None, C + (1 << 20), C + (2 << 20))
    assert call(A, 100, 0.1, ctypes.byref(bad), None, None) == EINVAL   # unsel missing
    alias = _lib.ZfSelection(A, C + 4096, C + (1 << 20), C + (2 << 20))
    assert call(A, 100, 0.1, ctypes.byref(alias), None, None) == EINVAL  # writes over scores
    assert call(None, 0, 0.1, ctypes.byref(s), ctypes.byref(kout), None) == OK
    assert kout.value == 0


def adam_args(**over):
    hp = _lib.ZfAdamHparams(1e-5, 0.9, 0.999, 1e-8, 0.0)
    args = dict(grad=A, n=8, m=64, ld=64, layout=RM, sel=sel(64, 6), k=6, P=B, M=B + (1 << 20),
                V=B + (2 << 20), lds=6, W=D, ldw=64, hp=hp, step=1, mode=0, src=None)
    args.update(over)
    return args


def call_adam(a):
    return LIB.zf_adam_selected(a["grad"], a["n"], a["m"], a["ld"], a["layout"],
                                ctypes.byref(a["sel"]),
                                a["k"], a["P"], a["M"], a["V"], a["lds"], a["W"], a["ldw"],
                                ctypes.byref(a["hp"]), a["step"], a["mode"],
                                ctypes.byref(a["src"]) if a["src"] is not None else None, None)


@pytest.mark.parametrize("over", [
    dict(step=0),
    dict(layout=2),
    dict(layout=CM),                               # [k][ld >= n] states: lds=6 < n=8
    dict(k=65),
    dict(lds=5),
    dict(ldw=63),
    dict(mode=7),
    dict(mode=1),                                  # remap without a source
    dict(M=B),                                     # exp_avg aliases master
    dict(W=A + 64),                                # weight overlaps gradient
    dict(P=None),
    dict(hp=_lib.ZfAdamHparams(1e-5, 1.0, 0.999, 1e-8, 0.0)),
    dict(hp=_lib.ZfAdamHparams(1e-5, 0.9, 0.999, -1.0, 0.0)),
    dict(hp=_lib.ZfAdamHparams(math.inf, 0.9, 0.999, 1e-8, 0.0)),
    dict(hp=_lib.ZfAdamHparams(1e-5, 0.9, 0.999, 1e-8, -0.1)),
])
def test_adam_validation(over):
    assert call_adam(adam_args(**over)) == EINVAL


def test_adam_remap_needs_previous_states():
    src = _lib.ZfStateSource(E, E + 4096, None, None, None, 0, None, 0)
    assert call_adam(adam_args(mode=1, src=src)) == EINVAL


def test_adam_empty_is_ok_without_device():
    assert call_adam(adam_args(n=0)) == OK
    assert call_adam(adam_args(k=0, P=None, M=None, V=None, lds=0, sel=sel(64, 0))) == OK


@pytest.mark.parametrize("sii,S", [(0, 4), (5, 4), (1, 0)])
def test_pack_validation(sii, S):
    s = sel(64, 6)
    assert LIB.zf_pack_accumulate(A, 8, 64, 64, RM, ctypes.byref(s), 6, B, 58, sii, S,
                                  None) == EINVAL


def test_pack_rejects_short_stride_and_alias():
    s = sel(64, 6)
    assert LIB.zf_pack_accumulate(A, 8, 64, 64, RM, ctypes.byref(s), 6, B, 57, 1, 4, None) == EINVAL
    assert LIB.zf_pack_accumulate(A, 8, 64, 64, RM, ctypes.byref(s), 6, A, 58, 1, 4, None) == EINVAL
    assert LIB.zf_pack_accumulate(A, 0, 64, 64, RM, ctypes.byref(s), 6, B, 58, 1, 4, None) == OK
    # channel-major packed buffer is [m-k][ld >= n]
    assert LIB.zf_pack_accumulate(A, 8, 64, 8, CM, ctypes.byref(s), 6, B, 7, 1, 4, None) == EINVAL


def test_unpack_validation():
    s = sel(64, 6)
    assert LIB.zf_unpack(B, 58, ctypes.byref(s), 6, 8, 64, RM, 1.0, B + 64, 64, None) == EINVAL
    assert LIB.zf_unpack(B, 58, ctypes.byref(s), 6, 8, 64, RM, 1.0, D, 63, None) == EINVAL
    assert LIB.zf_unpack(B, 58, None, 6, 8, 64, RM, 1.0, D, 64, None) == EINVAL
    assert LIB.zf_unpack(B, 58, ctypes.byref(s), 70, 8, 64, RM, 1.0, D, 64, None) == EINVAL
    assert LIB.zf_unpack(B, 8, ctypes.byref(s), 6, 8, 64, CM, 1.0, D, 7, None) == EINVAL


def test_update_fused_validation():
    s = sel(64, 6)
    hp = _lib.ZfAdamHparams(1e-5, 0.9, 0.999, 1e-8, 0.0)
    # accumulator aliasing the master states
    assert LIB.zf_update_fused(A, 8, 64, 64, RM, ctypes.byref(s), 6, B, B + (1 << 20),
                               B + (2 << 20), 6, D, 64, ctypes.byref(hp), 1, 0, None, B, 58, 1, 4,
                               None) == EINVAL
    assert LIB.zf_update_fused(A, 8, 64, 64, RM, ctypes.byref(s), 6, B, B + (1 << 20),
                               B + (2 << 20), 6, D, 64, ctypes.byref(hp), 1, 0, None, E, 58, 2, 1,
                               None) == EINVAL


def test_colnorm_noalloc_validation():
    """The allocation-free column scores reject on the host, before the
    static workspace is looked up: invalid arguments, and sizes whose
    workspace exceeds the static array."""
    n, m = 16384, 65536
    assert LIB.zf_colnorm_workspace_bytes(n, m, RM) == _lib.STATIC_SCRATCH_BYTES
    assert LIB.zf_colnorm_noalloc(A, n, m + 1, m + 8, RM, B, None) == EWS
    assert LIB.zf_colnorm_noalloc(A, 1 << 20, 4096, 4096, RM, B, None) == EWS  # 128 MiB
    assert LIB.zf_colnorm_noalloc(None, 4, 8, 8, RM, B, None) == EINVAL
    assert LIB.zf_colnorm_noalloc(A, 4, 8, 7, RM, B, None) == EINVAL  # ld < width
    assert LIB.zf_colnorm_noalloc(A, 4, 8, 8, 5, B, None) == EINVAL   # layout
    assert LIB.zf_colnorm_noalloc(A, 4, 8, 8, RM, None, None) == EINVAL
    assert LIB.zf_colnorm_noalloc(A, -1, 8, 8, RM, B, None) == EINVAL


def test_stream_probe_validation():
    """The measurement streams validate on the host before any launch."""
    P = LIB.zf_stream_probe
    assert "zf_stream_probe" in header_functions()
    assert P(3, A, B, 4096, 0, None) == EINVAL           # kind
    assert P(1, A, B, 0, 0, None) == EINVAL              # no bytes
    assert P(1, A, B, 4100, 0, None) == EINVAL           # not a multiple of 16
    assert P(1, A + 8, B, 4096, 0, None) == EINVAL       # src alignment
    assert P(1, A, B + 4, 4096, 0, None) == EINVAL       # dst alignment
    assert P(1, A, A + 1024, 4096, 0, None) == EINVAL    # overlapping copy
    assert P(0, None, B, 4096, 0, None) == EINVAL        # read without a source
    assert P(2, None, None, 4096, 0, None) == EINVAL     # rmw without a buffer
    assert P(1, A, B, 1 << 62, 0, None) == EINVAL        # too many blocks
    assert P(2, None, B, 4096 * (1 << 24), 0, None) == EINVAL   # 2^32 work-items: one too many


def test_plan_validation():
    h = ctypes.c_void_p()
    nb = ctypes.c_size_t()
    mem = 1 << 20  # a 256-aligned stand-in address: never reached, the descriptors fail first
    assert LIB.zf_plan_query(None, 1, ctypes.byref(nb)) == EINVAL
    assert LIB.zf_plan_create(None, 1, mem, 1 << 20, None, ctypes.byref(h)) == EINVAL
    arr = (_lib.ZfMatrix * 1)()
    assert LIB.zf_plan_query(arr, 0, ctypes.byref(nb)) == EINVAL
    assert LIB.zf_plan_create(arr, 0, mem, 1 << 20, None, ctypes.byref(h)) == EINVAL
    arr[0].n, arr[0].m, arr[0].k = 4, 4, 5          # k > m
    assert LIB.zf_plan_query(arr, 1, ctypes.byref(nb)) == EINVAL
    assert LIB.zf_plan_create(arr, 1, mem, 1 << 20, None, ctypes.byref(h)) == EINVAL
    arr2 = (_lib.ZfMatrix * 2)()
    arr2[0].n, arr2[0].m, arr2[0].k, arr2[0].layout = 0, 4, 1, RM
    arr2[1].n, arr2[1].m, arr2[1].k, arr2[1].layout = 0, 4, 1, CM   # mixed layouts
    assert LIB.zf_plan_query(arr2, 2, ctypes.byref(nb)) == EINVAL
    assert LIB.zf_plan_create(arr2, 2, mem, 1 << 20, None, ctypes.byref(h)) == EINVAL
    # valid descriptors (empty matrices): the size query succeeds on the host,
    # and create rejects missing, misaligned or too small device memory
    # before enqueueing anything
    ok = (_lib.ZfMatrix * 2)()
    ok[0].n, ok[0].m, ok[0].k, ok[0].layout = 0, 4, 1, RM
    ok[1].n, ok[1].m, ok[1].k, ok[1].layout = 0, 9, 2, RM
    assert LIB.zf_plan_query(ok, 2, ctypes.byref(nb)) == 0 and nb.value >= 256
    assert LIB.zf_plan_query(ok, 2, None) == EINVAL
    assert LIB.zf_plan_create(ok, 2, None, nb.value, None, ctypes.byref(h)) == EINVAL
    assert LIB.zf_plan_create(ok, 2, mem + 8, nb.value, None, ctypes.byref(h)) == EINVAL
    assert LIB.zf_plan_create(ok, 2, mem, nb.value - 1, None, ctypes.byref(h)) == EWS
    assert LIB.zf_plan_create(ok, 2, mem, nb.value, None, None) == EINVAL
    assert LIB.zf_plan_colnorm(None, None) == EINVAL
    assert LIB.zf_plan_update(None, None, 1, 0, 1, 1, 1, 1, None) == EINVAL
    hp = _lib.ZfAdamHparams(1e-5, 0.9, 0.999, 1e-8, 0.0)
    assert LIB.zf_plan_update_zen(None, ctypes.byref(hp), 1, 0, 1, 4, 1.0, None, None) == EINVAL
    assert _lib.ZEN_TOTALS_BYTES == 40
    assert LIB.zf_plan_device_bytes(None) == 0
    LIB.zf_plan_destroy(None)


def test_plan_entry_points_reject_a_missing_plan():
    """The deferred hand-over and the device-driven Zen-auto calls (with and
    without deferred packing) validate on the host: no plan, no state, a bad
    count or scale give ZF_EINVAL and nothing is enqueued (no GPU is
    touched)."""
    hp = _lib.ZfAdamHparams(1e-5, 0.9, 0.999, 1e-8, 0.0)
    hs = (ctypes.c_void_p * 16)()
    for n_earlier in (0, 1, 15, 16):
        assert LIB.zf_plan_update_handover_deferred(None, ctypes.byref(hp), 2, hs, n_earlier,
                                                    0.5, None) == EINVAL
    assert LIB.zf_plan_update_handover_deferred(None, None, 2, None, 1, float("nan"),
                                                None) == EINVAL
    assert LIB.zf_plan_update_zen_device(None, ctypes.byref(hp), 1, 0, 4, 0, 1.0, None, None,
                                         None) == EINVAL
    assert LIB.zf_plan_handover_zen(None, None, None) == EINVAL
    for n_earlier in (0, 1, 15, 16, -1):
        assert LIB.zf_plan_update_zen_deferred(None, ctypes.byref(hp), 1, 0, 4, hs, n_earlier,
                                               2, 1.0, None, None, None) == EINVAL
        assert LIB.zf_plan_handover_zen_deferred(None, hs, n_earlier, None, None) == EINVAL
    for name in ("zf_plan_update_handover_deferred", "zf_plan_update_zen_device",
                 "zf_plan_handover_zen", "zf_plan_update_zen_deferred",
                 "zf_plan_handover_zen_deferred"):
        assert name in header_functions()


def test_rowmajor_stage_stride_rule():
    """The row-major bf16 first-step stage needs 16-byte rows: a stride that
    is a multiple of 8 elements and a 16-byte aligned base.  A single row
    never uses its stride (the binding passes its width), so a one-row
    matrix of any width is accepted."""
    nb = ctypes.c_size_t()

    def query(n, m, ld_stage, stage=0x200000):
        arr = (_lib.ZfMatrix * 1)()
        x = arr[0]
        x.n, x.m, x.k, x.layout = n, m, 1, RM
        x.grad, x.ld_grad = 0x100000, 16
        x.acc_first, x.ld_acc_first = stage, ld_stage
        return LIB.zf_plan_query(arr, 1, ctypes.byref(nb))
    assert query(1, 9, 9) == 0 and query(1, 1, 1) == 0
    assert query(2, 9, 9) == EINVAL and query(2, 9, 16) == 0
    assert query(1, 9, 9, stage=0x200008) == EINVAL   # base alignment


def test_offload_and_handover_entry_points_validate_on_the_host():
    hp = _lib.ZfAdamHparams(1e-5, 0.9, 0.999, 1e-8, 0.0)
    s = _lib.ZfSelection()
    # no selection struct / null weights with data to write
    assert LIB.zf_scatter_weights(None, 8, None, 1, 4, 8, RM, None, 8, None) == EINVAL
    assert LIB.zf_scatter_weights(None, 8, ctypes.byref(s), 1, 4, 8, 7, None, 8, None) == EINVAL
    # fused hand-over: an output is required when there is data; k > m; bad layout
    assert LIB.zf_update_fused_handover(None, 4, 8, 8, RM, ctypes.byref(s), 1, None, None, None,
                                        1, None, 8, ctypes.byref(hp), 1, 0, None, None, 7, 1, 4,
                                        1.0, None, 8, None) == EINVAL
    assert LIB.zf_update_fused_handover(None, 0, 0, 0, RM, ctypes.byref(s), 0, None, None, None,
                                        0, None, 0, ctypes.byref(hp), 1, 0, None, None, 0, 1, 4,
                                        1.0, None, 0, None) == 0  # nothing to do
    assert LIB.zf_plan_update_handover(None, ctypes.byref(hp), 1, 0, 1, 4, 1.0, None) == EINVAL
    assert LIB.zf_plan_scatter_weights(None, None) == EINVAL
