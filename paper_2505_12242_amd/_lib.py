"""ctypes binding of libzf (include/zf.h).

Argument marshalling only: tensors are checked for dtype, device and
row-major layout, then their device addresses and row strides are passed to
the C ABI; every step of the path runs in the HIP kernels.  Importing this
module raises if libzf.so has not been built -- there is no fallback.
"""

from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import List, Optional, Sequence

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libzf.so")

ZF_OK, ZF_EINVAL, ZF_EWORKSPACE, ZF_EHIP, ZF_ENOMEM = 0, 1, 2, 3, 4
STATES_INPLACE, STATES_REMAP, STATES_INIT = 0, 1, 2
# Storage layouts (zf_layout).  A logical n x m matrix (n outputs, m input
# channels) is an [n, ld] tensor in ROW_MAJOR and an [m, ld] tensor (its
# transpose) in CHANNEL_MAJOR; compact states are [n, k] / [k, n] and the
# packed buffer [n, m-k] / [m-k, n] accordingly.
ROW_MAJOR, CHANNEL_MAJOR = 0, 1

c_i64, c_i32, c_dbl, c_flt, c_vp, c_sz = (ctypes.c_int64, ctypes.c_int32, ctypes.c_double,
                                          ctypes.c_float, ctypes.c_void_p, ctypes.c_size_t)


class ZfAdamHparams(ctypes.Structure):
    _fields_ = [("lr", c_dbl), ("beta1", c_dbl), ("beta2", c_dbl), ("eps", c_dbl),
                ("weight_decay", c_dbl)]


class ZfSelection(ctypes.Structure):
    _fields_ = [("sel_idx", c_vp), ("unsel_idx", c_vp), ("sel_mask", c_vp), ("sel_prefix", c_vp)]


class ZfStateSource(ctypes.Structure):
    _fields_ = [("prev_mask", c_vp), ("prev_prefix", c_vp), ("prev_master", c_vp),
                ("prev_exp_avg", c_vp), ("prev_exp_avg_sq", c_vp), ("ld_prev", c_i64),
                ("init_master", c_vp), ("ld_init", c_i64),
                ("store_master", c_vp), ("store_exp_avg", c_vp), ("store_exp_avg_sq", c_vp),
                ("ld_store", c_i64), ("pend_acc", c_vp), ("ld_pend", c_i64)]


class ZfMatrix(ctypes.Structure):
    _fields_ = [("n", c_i64), ("m", c_i64), ("k", c_i64), ("layout", c_i32),
                ("grad", c_vp), ("ld_grad", c_i64),
                ("weight", c_vp), ("ld_weight", c_i64),
                ("master", c_vp), ("exp_avg", c_vp), ("exp_avg_sq", c_vp), ("ld_state", c_i64),
                ("acc", c_vp), ("ld_acc", c_i64),
                ("norms_sq", c_vp),
                ("sel", ZfSelection),
                ("unpacked", c_vp), ("ld_unpacked", c_i64),
                ("src", ZfStateSource),
                ("sel_sq", c_vp), ("acc_sq", c_vp),
                ("weight_cols", c_vp), ("ld_weight_cols", c_i64),
                ("acc_first", c_vp), ("ld_acc_first", c_i64)]


class ZfZenTotals(ctypes.Structure):
    _fields_ = [("sum_sel", c_dbl), ("sum_acc", c_dbl), ("k_total", c_i64), ("u_total", c_i64),
                ("trigger", c_i32), ("pad", c_i32)]


# (name, restype, argtypes) of every exported entry point of include/zf.h.
SIGNATURES = [
    ("zf_status_string", ctypes.c_char_p, [ctypes.c_int]),
    ("zf_last_hip_error", ctypes.c_int, []),
    ("zf_k_from_ratio", c_i64, [c_dbl, c_i64]),
    ("zf_colnorm_workspace_bytes", c_sz, [c_i64, c_i64, c_i32]),
    ("zf_colnorm", ctypes.c_int, [c_vp, c_i64, c_i64, c_i64, c_i32, c_vp, c_vp, c_sz, c_vp]),
    ("zf_colnorm_noalloc", ctypes.c_int, [c_vp, c_i64, c_i64, c_i64, c_i32, c_vp, c_vp]),
    ("zf_stream_probe", ctypes.c_int, [c_i32, c_vp, c_vp, c_sz, ctypes.c_uint32, c_vp]),
    ("zf_topk_select", ctypes.c_int,
     [c_vp, c_i64, c_dbl, ctypes.POINTER(ZfSelection), ctypes.POINTER(c_i64), c_vp]),
    ("zf_adam_selected", ctypes.c_int,
     [c_vp, c_i64, c_i64, c_i64, c_i32, ctypes.POINTER(ZfSelection), c_i64, c_vp, c_vp, c_vp, c_i64,
      c_vp, c_i64, ctypes.POINTER(ZfAdamHparams), c_i64, c_i32, ctypes.POINTER(ZfStateSource),
      c_vp]),
    ("zf_pack_accumulate", ctypes.c_int,
     [c_vp, c_i64, c_i64, c_i64, c_i32, ctypes.POINTER(ZfSelection), c_i64, c_vp, c_i64, c_i64, c_i64,
      c_vp]),
    ("zf_update_fused", ctypes.c_int,
     [c_vp, c_i64, c_i64, c_i64, c_i32, ctypes.POINTER(ZfSelection), c_i64, c_vp, c_vp, c_vp, c_i64,
      c_vp, c_i64, ctypes.POINTER(ZfAdamHparams), c_i64, c_i32, ctypes.POINTER(ZfStateSource),
      c_vp, c_i64, c_i64, c_i64, c_vp]),
    ("zf_update_fused_handover", ctypes.c_int,
     [c_vp, c_i64, c_i64, c_i64, c_i32, ctypes.POINTER(ZfSelection), c_i64, c_vp, c_vp, c_vp, c_i64,
      c_vp, c_i64, ctypes.POINTER(ZfAdamHparams), c_i64, c_i32, ctypes.POINTER(ZfStateSource),
      c_vp, c_i64, c_i64, c_i64, c_flt, c_vp, c_i64, c_vp]),
    ("zf_unpack", ctypes.c_int,
     [c_vp, c_i64, ctypes.POINTER(ZfSelection), c_i64, c_i64, c_i64, c_i32, c_flt, c_vp, c_i64,
      c_vp]),
    ("zf_plan_query", ctypes.c_int, [ctypes.POINTER(ZfMatrix), c_i32, ctypes.POINTER(c_sz)]),
    ("zf_plan_create", ctypes.c_int,
     [ctypes.POINTER(ZfMatrix), c_i32, c_vp, c_sz, c_vp, ctypes.POINTER(c_vp)]),
    ("zf_plan_destroy", None, [c_vp]),
    ("zf_plan_device_bytes", c_sz, [c_vp]),
    ("zf_plan_colnorm", ctypes.c_int, [c_vp, c_vp]),
    ("zf_plan_topk_select", ctypes.c_int, [c_vp, c_vp]),
    ("zf_plan_colnorm_stage", ctypes.c_int, [c_vp, c_vp]),
    ("zf_plan_unpack_first", ctypes.c_int, [c_vp, c_flt, c_vp]),
    ("zf_plan_colnorm_handover", ctypes.c_int, [c_vp, c_flt, c_vp]),
    ("zf_plan_update_adam_handover", ctypes.c_int,
     [c_vp, ctypes.POINTER(ZfAdamHparams), c_i64, c_i32, c_vp]),
    ("zf_plan_update", ctypes.c_int,
     [c_vp, ctypes.POINTER(ZfAdamHparams), c_i64, c_i32, c_i64, c_i64, c_i32, c_i32, c_vp]),
    ("zf_plan_unpack", ctypes.c_int, [c_vp, c_flt, c_vp]),
    ("zf_host_adam_unselected", ctypes.c_int,
     [c_vp, c_i64, c_vp, c_i64, c_i64, c_i64, c_i32, c_flt, c_vp, c_vp, c_vp, c_i64, c_vp, c_i64,
      ctypes.POINTER(ZfAdamHparams), c_i64, c_i32]),
    ("zf_scatter_weights", ctypes.c_int,
     [c_vp, c_i64, ctypes.POINTER(ZfSelection), c_i64, c_i64, c_i64, c_i32, c_vp, c_i64, c_vp]),
    ("zf_plan_scatter_weights", ctypes.c_int, [c_vp, c_vp]),
    ("zf_plan_update_handover", ctypes.c_int,
     [c_vp, ctypes.POINTER(ZfAdamHparams), c_i64, c_i32, c_i64, c_i64, c_flt, c_vp]),
    ("zf_plan_update_zen", ctypes.c_int,
     [c_vp, ctypes.POINTER(ZfAdamHparams), c_i64, c_i32, c_i64, c_i64, c_dbl, c_vp, c_vp]),
    ("zf_plan_update_pending", ctypes.c_int,
     [c_vp, ctypes.POINTER(ZfAdamHparams), c_i64, c_i64, c_i64, c_flt, c_vp]),
    ("zf_plan_scatter_weights_skip_prev", ctypes.c_int, [c_vp, c_vp]),
    ("zf_plan_update_handover_deferred", ctypes.c_int,
     [c_vp, ctypes.POINTER(ZfAdamHparams), c_i64, ctypes.POINTER(c_vp), c_i32, c_flt, c_vp]),
    ("zf_plan_update_zen_device", ctypes.c_int,
     [c_vp, ctypes.POINTER(ZfAdamHparams), c_i64, c_i32, c_i64, c_i32, c_dbl, c_vp, c_vp, c_vp]),
    ("zf_plan_handover_zen", ctypes.c_int, [c_vp, c_vp, c_vp]),
    ("zf_plan_update_zen_deferred", ctypes.c_int,
     [c_vp, ctypes.POINTER(ZfAdamHparams), c_i64, c_i32, c_i64, ctypes.POINTER(c_vp), c_i32,
      c_i32, c_dbl, c_vp, c_vp, c_vp]),
    ("zf_plan_handover_zen_deferred", ctypes.c_int,
     [c_vp, ctypes.POINTER(c_vp), c_i32, c_vp, c_vp]),
    ("zf_plan_update_zen_pending", ctypes.c_int,
     [c_vp, ctypes.POINTER(ZfAdamHparams), c_i64, c_i64, c_i64, c_flt, c_dbl, c_vp, c_vp]),
]


def load(path: str = LIB_PATH) -> ctypes.CDLL:
    if not os.path.exists(path):
        raise RuntimeError(
            f"libzf.so is not built ({path} missing); run `python paper_2505_12242_amd/build.py`")
    lib = ctypes.CDLL(path)
    for name, res, args in SIGNATURES:
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    return lib


LIB = load()


class ZfError(RuntimeError):
    def __init__(self, fn: str, status: int):
        msg = LIB.zf_status_string(status).decode()
        if status == ZF_EHIP:
            msg += f" (hipError {LIB.zf_last_hip_error()})"
        super().__init__(f"{fn}: {msg}")
        self.status = status


def _check(fn: str, status: int) -> None:
    if status != ZF_OK:
        raise ZfError(fn, status)


# ---------------------------------------------------------------------------
# tensor marshalling
# ---------------------------------------------------------------------------

def _ptr(t: Optional[torch.Tensor]):
    return None if t is None or t.numel() == 0 else t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def _mat(t: torch.Tensor, dtype, name: str, rows: Optional[int] = None,
         cols: Optional[int] = None, device_ok: bool = False, host: bool = False) -> int:
    """Checks a row-major 2-D tensor and returns its row stride.  The tensor
    must live on a GPU; device_ok also accepts pinned host memory (which the
    kernels access in place); host requires a CPU tensor."""
    if t.dtype != dtype:
        raise TypeError(f"{name}: expected {dtype}, got {t.dtype}")
    if t.dim() != 2:
        raise ValueError(f"{name}: expected a 2-D tensor, got shape {tuple(t.shape)}")
    if rows is not None and t.shape[0] != rows:
        raise ValueError(f"{name}: expected {rows} rows, got {t.shape[0]}")
    if cols is not None and t.shape[1] != cols:
        raise ValueError(f"{name}: expected {cols} columns, got {t.shape[1]}")
    if t.numel():
        if host:
            if t.is_cuda:
                raise ValueError(f"{name}: must be a host (CPU) tensor")
        elif not (t.is_cuda or (device_ok and t.is_pinned())):
            raise ValueError(f"{name}: must live on a GPU" +
                             (" or in pinned host memory" if device_ok else ""))
    if t.shape[0] > 1 and t.shape[1] > 1 and t.stride(1) != 1:
        raise ValueError(f"{name}: rows must be contiguous (stride(1) == 1)")
    return t.stride(0) if t.shape[0] > 1 else t.shape[1]


def _logical(t: torch.Tensor, layout: int):
    """(n, m) of a matrix stored as tensor t in `layout`."""
    if layout not in (ROW_MAJOR, CHANNEL_MAJOR):
        raise ValueError(f"unknown layout {layout}")
    return (t.shape[0], t.shape[1]) if layout == ROW_MAJOR else (t.shape[1], t.shape[0])


def _stored(layout: int, rows_l: int, cols_l: int):
    """Tensor shape of a logical rows_l x cols_l matrix in `layout`."""
    return (rows_l, cols_l) if layout == ROW_MAJOR else (cols_l, rows_l)


def alloc_stored(layout: int, rows_l: int, cols_l: int, dtype=torch.float32,
                 device="cuda", pin_memory: bool = False) -> torch.Tensor:
    """Uninitialised storage of a logical rows_l x cols_l matrix in `layout`.
    Row-major rows are padded to a multiple of 16 bytes (the returned tensor
    is a view of the first cols_l columns), which lets the row-major update
    move packed buffers, compact states and hand-over rows 16 bytes at a
    time; channel-major storage is dense.  pin_memory: pinned host memory."""
    kw = dict(dtype=dtype, pin_memory=True) if pin_memory else dict(dtype=dtype, device=device)
    if layout != ROW_MAJOR:
        return torch.empty(*_stored(layout, rows_l, cols_l), **kw)
    per = 16 // torch.empty(0, dtype=dtype).element_size()
    ld = max(per, -(-cols_l // per) * per)
    return torch.empty(rows_l, ld, **kw)[:, :cols_l]


_HIP = None


def _hip():
    """The HIP runtime, for the few calls the binding makes itself (pinned
    host allocation, asynchronous copies of it)."""
    global _HIP
    if _HIP is None:
        lib = ctypes.CDLL("libamdhip64.so")
        lib.hipHostMalloc.restype = ctypes.c_int
        lib.hipHostMalloc.argtypes = [ctypes.POINTER(c_vp), c_sz, ctypes.c_uint]
        lib.hipHostFree.restype = ctypes.c_int
        lib.hipHostFree.argtypes = [c_vp]
        lib.hipMemcpyAsync.restype = ctypes.c_int
        lib.hipMemcpyAsync.argtypes = [c_vp, c_vp, c_sz, ctypes.c_int, c_vp]
        _HIP = lib
    return _HIP


def copy_async(dst: torch.Tensor, src: torch.Tensor, stream) -> None:
    """dst <- src as one hipMemcpyAsync on `stream` (a torch stream): both
    dense, the same size in bytes, either on the GPU or in pinned host
    memory.  Used for PinnedArena tensors, which torch does not recognise as
    pinned (its own non_blocking copies would turn synchronous)."""
    n = dst.numel() * dst.element_size()
    if src.numel() * src.element_size() != n or not (dst.is_contiguous() and src.is_contiguous()):
        raise ValueError("copy_async: dense tensors of the same size expected")
    if n == 0:
        return
    err = _hip().hipMemcpyAsync(dst.data_ptr(), src.data_ptr(), n, 4,  # hipMemcpyDefault
                                stream.cuda_stream)
    if err != 0:
        raise RuntimeError(f"hipMemcpyAsync failed (hipError {err})")


class PinnedArena:
    """Pinned host memory of exactly the size asked for, handed out as CPU
    tensors.  torch's pinned allocator rounds every allocation up to a
    power of two, which for the offloaded optimizer's store and staging of a
    whole gradient set (tens of GB each) wastes up to half of the pinned
    memory a process is granted.  The arena allocates hipHostMalloc chunks
    of at most CHUNK bytes (a single pinned allocation is limited well below
    the total a process may pin) and places tensors in them back to back.
    torch does not see these tensors as pinned: copy them with copy_async.
    The caller frees the arena (free()) once no GPU work and no host thread
    uses its tensors."""

    CHUNK = 32 << 30

    def __init__(self, nbytes: int):
        self.total = int(nbytes)
        self.allocated = 0
        self.chunks = []  # (pointer, size, base tensor)
        self.used = 0     # bytes used in the last chunk

    @staticmethod
    def bytes_for(shape, dtype) -> int:
        n = 1
        for x in shape:
            n *= int(x)
        return n * torch.empty(0, dtype=dtype).element_size() + 256

    @staticmethod
    def stored_shape(layout: int, rows_l: int, cols_l: int, dtype):
        """Dense shape alloc_stored uses for a logical matrix (row-major rows
        padded to 16 bytes)."""
        if layout != ROW_MAJOR:
            return _stored(layout, rows_l, cols_l)
        per = 16 // torch.empty(0, dtype=dtype).element_size()
        return (rows_l, max(per, -(-cols_l // per) * per))

    def _new_chunk(self, need: int) -> None:
        size = max(need, min(self.CHUNK, max(self.total - self.allocated, need)), 256)
        ptr = c_vp()
        err = _hip().hipHostMalloc(ctypes.byref(ptr), size, 0)
        if err != 0 or not ptr.value:
            raise MemoryError(f"hipHostMalloc of {size / 1e9:.1f} GB failed after "
                              f"{self.allocated / 1e9:.1f} GB (hipError {err})")
        base = torch.frombuffer((ctypes.c_char * size).from_address(ptr.value), dtype=torch.uint8)
        self.chunks.append((ptr.value, size, base))
        self.allocated += size
        self.used = 0

    def take(self, shape, dtype) -> torch.Tensor:
        """A tensor of `shape` in the arena (256-byte aligned)."""
        n = self.bytes_for(shape, dtype) - 256
        off = (self.used + 255) & ~255
        if not self.chunks or off + n > self.chunks[-1][1]:
            self._new_chunk(n)
            off = 0
        self.used = off + n
        return self.chunks[-1][2][off: off + n].view(dtype).view(*shape)

    def take_stored(self, layout: int, rows_l: int, cols_l: int, dtype) -> torch.Tensor:
        """alloc_stored(..., pin_memory=True) in the arena."""
        t = self.take(self.stored_shape(layout, rows_l, cols_l, dtype), dtype)
        return t if layout != ROW_MAJOR else t[:, :cols_l]

    def free(self) -> None:
        for ptr, _, _ in self.chunks:
            _hip().hipHostFree(ptr)
        self.chunks = []
        self.allocated = 0


def padded_block(t: torch.Tensor) -> torch.Tensor:
    """The rows of a 2-D view including their padding (a dense tensor over
    the same memory), e.g. for one contiguous copy of a padded buffer."""
    if t.dim() != 2 or t.shape[0] == 0 or t.stride(1) != 1:
        return t
    return t.as_strided((t.shape[0], t.stride(0)), (t.stride(0), 1))


def _lmat(t, dtype, name, layout, rows_l=None, cols_l=None, **kw) -> int:
    r, c = (rows_l, cols_l) if layout == ROW_MAJOR else (cols_l, rows_l)
    return _mat(t, dtype, name, r, c, **kw)


def _vec(t: torch.Tensor, dtype, name: str, size: int) -> None:
    if t.dtype != dtype or t.dim() != 1 or t.shape[0] != size:
        raise ValueError(f"{name}: expected a [{size}] {dtype} tensor, got "
                         f"{tuple(t.shape)} {t.dtype}")
    if size and (not t.is_cuda or not t.is_contiguous()):
        raise ValueError(f"{name}: must be a contiguous GPU tensor")


@dataclass
class AdamHparams:
    lr: float = 1e-5
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-8
    weight_decay: float = 0.0

    def as_c(self) -> ZfAdamHparams:
        return ZfAdamHparams(self.lr, self.beta1, self.beta2, self.eps, self.weight_decay)


class Selection:
    """Device buffers of one selection of k out of m columns."""

    def __init__(self, m: int, k: int, device=None):
        device = device if device is not None else torch.device("cuda")
        words = (m + 63) // 64
        self.m, self.k = m, k
        self.sel_idx = torch.empty(k, dtype=torch.int32, device=device)
        self.unsel_idx = torch.empty(m - k, dtype=torch.int32, device=device)
        self.mask = torch.empty(words, dtype=torch.int64, device=device)  # uint64 bit patterns
        self.prefix = torch.empty(words, dtype=torch.int32, device=device)

    def as_c(self) -> ZfSelection:
        return ZfSelection(_ptr(self.sel_idx), _ptr(self.unsel_idx), _ptr(self.mask),
                           _ptr(self.prefix))


def k_from_ratio(ratio: float, m: int) -> int:
    k = LIB.zf_k_from_ratio(float(ratio), int(m))
    if k < 0:
        raise ValueError("ratio must lie in [0, 1] and m >= 0")
    return k


def colnorm_workspace_bytes(n: int, m: int, layout: int = ROW_MAJOR) -> int:
    return LIB.zf_colnorm_workspace_bytes(n, m, layout)


def colnorm(grad: torch.Tensor, out: Optional[torch.Tensor] = None,
            workspace: Optional[torch.Tensor] = None, layout: int = ROW_MAJOR,
            stream=None) -> torch.Tensor:
    n, m = _logical(grad, layout)
    ld = _mat(grad, torch.bfloat16, "grad")
    if out is None:
        out = torch.empty(m, dtype=torch.float32, device=grad.device)
    _vec(out, torch.float32, "out", m)
    need = colnorm_workspace_bytes(n, m, layout)
    if workspace is None:
        workspace = torch.empty(max(need, 8), dtype=torch.uint8, device=grad.device)
    _check("zf_colnorm", LIB.zf_colnorm(_ptr(grad), n, m, ld, layout, _ptr(out),
                                        _ptr(workspace), workspace.numel(), _stream(stream)))
    return out


STATIC_SCRATCH_BYTES = 32 << 20  # ZF_STATIC_SCRATCH_BYTES


def colnorm_noalloc(grad: torch.Tensor, out: torch.Tensor, layout: int = ROW_MAJOR,
                    stream=None) -> torch.Tensor:
    """zf_colnorm_noalloc: the column scores with the library's static
    per-GPU workspace; `out` ([m] fp32 on the GPU) is caller-provided, so
    the call allocates nothing."""
    n, m = _logical(grad, layout)
    ld = _mat(grad, torch.bfloat16, "grad")
    _vec(out, torch.float32, "out", m)
    _check("zf_colnorm_noalloc", LIB.zf_colnorm_noalloc(_ptr(grad), n, m, ld, layout, _ptr(out),
                                                        _stream(stream)))
    return out


PROBE_READ, PROBE_COPY, PROBE_RMW = 0, 1, 2


def stream_probe(kind: int, src: Optional[torch.Tensor], dst: torch.Tensor, nbytes: int,
                 key: int = 0, stream=None) -> None:
    """One reference streaming pass of zf_measure.h (zf_stream_probe) over
    the first `nbytes` of src / dst (GPU tensors)."""
    for t, name in ((src, "src"), (dst, "dst")):
        if t is not None and (not t.is_cuda or not t.is_contiguous()):
            raise ValueError(f"{name}: expected a contiguous GPU tensor")
    if src is not None and src.numel() * src.element_size() < nbytes and kind != PROBE_RMW:
        raise ValueError("src smaller than nbytes")
    if kind != PROBE_READ and dst.numel() * dst.element_size() < nbytes:
        raise ValueError("dst smaller than nbytes")
    _check("zf_stream_probe", LIB.zf_stream_probe(int(kind), _ptr(src), _ptr(dst), int(nbytes),
                                                  int(key) & 0xFFFFFFFF, _stream(stream)))


def topk_select(norms: torch.Tensor, ratio: float, out: Optional[Selection] = None,
                stream=None) -> Selection:
    m = norms.shape[0]
    k = k_from_ratio(ratio, m)
    _vec(norms, torch.float32, "norms", m)
    if out is None:
        out = Selection(m, k, norms.device)
    if out.m != m or out.k != k:
        raise ValueError(f"selection buffers are for m={out.m}, k={out.k}; need m={m}, k={k}")
    c_sel = out.as_c()
    k_out = c_i64(-1)
    _check("zf_topk_select", LIB.zf_topk_select(_ptr(norms), m, float(ratio), ctypes.byref(c_sel),
                                                ctypes.byref(k_out), _stream(stream)))
    return out


@dataclass
class StateSource:
    """Where the selected columns' states come from (see zf_state_mode).
    Tensors are stored in the same layout as the call that uses them."""
    prev: Optional[Selection] = None
    prev_master: Optional[torch.Tensor] = None
    prev_exp_avg: Optional[torch.Tensor] = None
    prev_exp_avg_sq: Optional[torch.Tensor] = None
    init_master: Optional[torch.Tensor] = None
    # full-state store (swap-in / swap-out); device or pinned host tensors
    store_master: Optional[torch.Tensor] = None
    store_exp_avg: Optional[torch.Tensor] = None
    store_exp_avg_sq: Optional[torch.Tensor] = None
    # packed sums of the interval that ended just before a refresh, under the
    # previous selection (the deferred update the store still owes; read by
    # Plan.update_pending only)
    pend_acc: Optional[torch.Tensor] = None

    def as_c(self) -> ZfStateSource:
        ld_prev = 0
        if self.prev_master is not None:
            ld_prev = _mat(self.prev_master, torch.float32, "prev_master")
            if (_mat(self.prev_exp_avg, torch.float32, "prev_exp_avg") != ld_prev
                    or _mat(self.prev_exp_avg_sq, torch.float32, "prev_exp_avg_sq") != ld_prev):
                raise ValueError("previous states must share one row stride")
        ld_init = 0
        if self.init_master is not None:
            ld_init = _mat(self.init_master, torch.float32, "init_master")
        ld_store = 0
        if self.store_master is not None:
            ld_store = _mat(self.store_master, torch.float32, "store_master", device_ok=True)
            if (_mat(self.store_exp_avg, torch.float32, "store_exp_avg", device_ok=True) != ld_store
                    or _mat(self.store_exp_avg_sq, torch.float32, "store_exp_avg_sq",
                            device_ok=True) != ld_store):
                raise ValueError("the store's three arrays must share one row stride")
        ld_pend = 0
        if self.pend_acc is not None:
            ld_pend = _mat(self.pend_acc, torch.float32, "pend_acc", device_ok=True)
        return ZfStateSource(
            _ptr(self.prev.mask) if self.prev else None,
            _ptr(self.prev.prefix) if self.prev else None,
            _ptr(self.prev_master), _ptr(self.prev_exp_avg), _ptr(self.prev_exp_avg_sq), ld_prev,
            _ptr(self.init_master), ld_init,
            _ptr(self.store_master), _ptr(self.store_exp_avg), _ptr(self.store_exp_avg_sq),
            ld_store, _ptr(self.pend_acc), ld_pend)


def _states(n, k, master, exp_avg, exp_avg_sq, layout):
    ld = _lmat(master, torch.float32, "master", layout, n, k)
    if (_lmat(exp_avg, torch.float32, "exp_avg", layout, n, k) != ld
            or _lmat(exp_avg_sq, torch.float32, "exp_avg_sq", layout, n, k) != ld):
        raise ValueError("master, exp_avg and exp_avg_sq must share one row stride")
    return ld


def adam_selected(grad, sel: Selection, master, exp_avg, exp_avg_sq, weight, hp: AdamHparams,
                  step: int, mode: int = STATES_INPLACE, src: Optional[StateSource] = None,
                  layout: int = ROW_MAJOR, stream=None) -> None:
    n, m = _logical(grad, layout)
    ldg = _mat(grad, torch.bfloat16, "grad")
    lds = _states(n, sel.k, master, exp_avg, exp_avg_sq, layout)
    ldw = _lmat(weight, torch.bfloat16, "weight", layout, n, m)
    c_sel, c_hp = sel.as_c(), hp.as_c()
    c_src = src.as_c() if src is not None else None
    _check("zf_adam_selected", LIB.zf_adam_selected(
        _ptr(grad), n, m, ldg, layout, ctypes.byref(c_sel), sel.k, _ptr(master), _ptr(exp_avg),
        _ptr(exp_avg_sq), lds, _ptr(weight), ldw, ctypes.byref(c_hp), step, mode,
        ctypes.byref(c_src) if c_src is not None else None, _stream(stream)))


def pack_accumulate(grad, sel: Selection, acc, step_in_interval: int, accum_interval: int,
                    layout: int = ROW_MAJOR, stream=None) -> None:
    n, m = _logical(grad, layout)
    ldg = _mat(grad, torch.bfloat16, "grad")
    lda = _lmat(acc, torch.float32, "acc", layout, n, m - sel.k)
    c_sel = sel.as_c()
    _check("zf_pack_accumulate", LIB.zf_pack_accumulate(
        _ptr(grad), n, m, ldg, layout, ctypes.byref(c_sel), sel.k, _ptr(acc), lda,
        step_in_interval, accum_interval, _stream(stream)))


def update_fused(grad, sel: Selection, master, exp_avg, exp_avg_sq, weight, hp: AdamHparams,
                 step: int, acc, step_in_interval: int, accum_interval: int,
                 mode: int = STATES_INPLACE, src: Optional[StateSource] = None,
                 layout: int = ROW_MAJOR, stream=None) -> None:
    n, m = _logical(grad, layout)
    ldg = _mat(grad, torch.bfloat16, "grad")
    lds = _states(n, sel.k, master, exp_avg, exp_avg_sq, layout)
    ldw = _lmat(weight, torch.bfloat16, "weight", layout, n, m)
    lda = _lmat(acc, torch.float32, "acc", layout, n, m - sel.k)
    c_sel, c_hp = sel.as_c(), hp.as_c()
    c_src = src.as_c() if src is not None else None
    _check("zf_update_fused", LIB.zf_update_fused(
        _ptr(grad), n, m, ldg, layout, ctypes.byref(c_sel), sel.k, _ptr(master), _ptr(exp_avg),
        _ptr(exp_avg_sq), lds, _ptr(weight), ldw, ctypes.byref(c_hp), step, mode,
        ctypes.byref(c_src) if c_src is not None else None, _ptr(acc), lda, step_in_interval,
        accum_interval, _stream(stream)))


def update_fused_handover(grad, sel: Selection, master, exp_avg, exp_avg_sq, weight,
                          hp: AdamHparams, step: int, acc, step_in_interval: int,
                          accum_interval: int, scale: float, out: Optional[torch.Tensor] = None,
                          mode: int = STATES_INPLACE, src: Optional[StateSource] = None,
                          layout: int = ROW_MAJOR, stream=None) -> torch.Tensor:
    """The last step of an interval in one pass: Adam on the selected columns
    and out = scale * (A + G) at the unselected ones, +0.0 at the selected
    (zf_update_fused_handover); A is only read."""
    n, m = _logical(grad, layout)
    ldg = _mat(grad, torch.bfloat16, "grad")
    lds = _states(n, sel.k, master, exp_avg, exp_avg_sq, layout)
    ldw = _lmat(weight, torch.bfloat16, "weight", layout, n, m)
    lda = _lmat(acc, torch.float32, "acc", layout, n, m - sel.k)
    if out is None:
        out = alloc_stored(layout, n, m, torch.float32, grad.device)
    ldo = _lmat(out, torch.float32, "out", layout, n, m)
    c_sel, c_hp = sel.as_c(), hp.as_c()
    c_src = src.as_c() if src is not None else None
    _check("zf_update_fused_handover", LIB.zf_update_fused_handover(
        _ptr(grad), n, m, ldg, layout, ctypes.byref(c_sel), sel.k, _ptr(master), _ptr(exp_avg),
        _ptr(exp_avg_sq), lds, _ptr(weight), ldw, ctypes.byref(c_hp), step, mode,
        ctypes.byref(c_src) if c_src is not None else None, _ptr(acc), lda, step_in_interval,
        accum_interval, float(scale), _ptr(out), ldo, _stream(stream)))
    return out


def unpack(acc, sel: Selection, scale: float = 1.0, out: Optional[torch.Tensor] = None,
           layout: int = ROW_MAJOR, stream=None) -> torch.Tensor:
    m = sel.m
    n = acc.shape[0] if layout == ROW_MAJOR else acc.shape[1]
    lda = _lmat(acc, torch.float32, "acc", layout, n, m - sel.k)
    if out is None:
        out = alloc_stored(layout, n, m, torch.float32, acc.device)
    ldo = _lmat(out, torch.float32, "out", layout, n, m)
    c_sel = sel.as_c()
    _check("zf_unpack", LIB.zf_unpack(_ptr(acc), lda, ctypes.byref(c_sel), sel.k, n, m, layout,
                                      float(scale), _ptr(out), ldo, _stream(stream)))
    return out


def host_adam_unselected(acc: torch.Tensor, unsel_idx: torch.Tensor, n: int, m: int, k: int,
                         scale: float, master: torch.Tensor, exp_avg: torch.Tensor,
                         exp_avg_sq: torch.Tensor, weight_cols: torch.Tensor, hp: AdamHparams,
                         step: int, layout: int = ROW_MAJOR, nthreads: int = 0) -> None:
    """The deferred host update (zf_host_adam_unselected): every argument is
    a host (CPU) tensor; runs on `nthreads` host threads (0 = all)."""
    u = m - k
    lda = _lmat(acc, torch.float32, "acc", layout, n, u, host=True) if n * u else max(u, n, 1)
    if unsel_idx.is_cuda or unsel_idx.dtype != torch.int32 or unsel_idx.numel() != u \
            or not unsel_idx.is_contiguous():
        raise ValueError(f"unsel_idx: expected a contiguous [{u}] int32 host tensor")
    for t, name in ((acc, "acc"), (master, "master"), (exp_avg, "exp_avg"),
                    (exp_avg_sq, "exp_avg_sq"), (weight_cols, "weight_cols")):
        if t.is_cuda:
            raise ValueError(f"{name}: must be a host (CPU) tensor")
    lds = _lmat(master, torch.float32, "master", layout, n, m, host=True)
    if (_lmat(exp_avg, torch.float32, "exp_avg", layout, n, m, host=True) != lds
            or _lmat(exp_avg_sq, torch.float32, "exp_avg_sq", layout, n, m, host=True) != lds):
        raise ValueError("master, exp_avg and exp_avg_sq must share one row stride")
    ldw = (_lmat(weight_cols, torch.bfloat16, "weight_cols", layout, n, u, host=True)
           if n * u else max(u, n, 1))
    c_hp = hp.as_c()
    _check("zf_host_adam_unselected", LIB.zf_host_adam_unselected(
        _ptr(acc), lda, _ptr(unsel_idx), n, m, k, layout, float(scale), _ptr(master),
        _ptr(exp_avg), _ptr(exp_avg_sq), lds, _ptr(weight_cols), ldw, ctypes.byref(c_hp),
        int(step), int(nthreads)))


def scatter_weights(weight_cols: torch.Tensor, sel: Selection, weight: torch.Tensor,
                    layout: int = ROW_MAJOR, stream=None) -> None:
    """W[:, unsel] = weight_cols (zf_scatter_weights); weight_cols may be a
    device tensor or a pinned host tensor."""
    n, m = _logical(weight, layout)
    ldw = _mat(weight, torch.bfloat16, "weight")
    r, c = _stored(layout, n, m - sel.k)
    ldc = (_mat(weight_cols, torch.bfloat16, "weight_cols", r, c, device_ok=True) if r * c
           else max(c, 1))
    c_sel = sel.as_c()
    _check("zf_scatter_weights", LIB.zf_scatter_weights(
        _ptr(weight_cols), ldc, ctypes.byref(c_sel), sel.k, n, m, layout, _ptr(weight), ldw,
        _stream(stream)))


# ---------------------------------------------------------------------------
# batched plans
# ---------------------------------------------------------------------------

@dataclass
class MatrixBuffers:
    """Device tensors of one matrix of a batch, all in `layout`; unused
    stages may be None."""
    grad: torch.Tensor
    k: int
    sel: Selection
    weight: Optional[torch.Tensor] = None
    master: Optional[torch.Tensor] = None
    exp_avg: Optional[torch.Tensor] = None
    exp_avg_sq: Optional[torch.Tensor] = None
    acc: Optional[torch.Tensor] = None
    norms: Optional[torch.Tensor] = None
    unpacked: Optional[torch.Tensor] = None
    src: Optional[StateSource] = None
    layout: int = ROW_MAJOR
    sel_sq: Optional[torch.Tensor] = None   # Zen-auto statistics, [k] fp32
    acc_sq: Optional[torch.Tensor] = None   # Zen-auto statistics, [m-k] fp32
    weight_cols: Optional[torch.Tensor] = None  # deferred update: bf16 unselected columns
    acc_first: Optional[torch.Tensor] = None  # channel-major: bf16 first-step stage, [m, n]

    def as_c(self) -> ZfMatrix:
        L = self.layout
        n, m = _logical(self.grad, L)
        x = ZfMatrix()
        x.n, x.m, x.k, x.layout = n, m, self.k, L
        x.grad, x.ld_grad = _ptr(self.grad), _mat(self.grad, torch.bfloat16, "grad")
        if self.weight is not None:
            x.weight = _ptr(self.weight)
            x.ld_weight = _lmat(self.weight, torch.bfloat16, "weight", L, n, m)
        if self.master is not None:
            x.master, x.exp_avg, x.exp_avg_sq = (_ptr(self.master), _ptr(self.exp_avg),
                                                 _ptr(self.exp_avg_sq))
            x.ld_state = _states(n, self.k, self.master, self.exp_avg, self.exp_avg_sq, L)
        if self.acc is not None:
            x.acc = _ptr(self.acc)
            x.ld_acc = _lmat(self.acc, torch.float32, "acc", L, n, m - self.k)
        if self.norms is not None:
            _vec(self.norms, torch.float32, "norms", m)
            x.norms_sq = _ptr(self.norms)
        x.sel = self.sel.as_c()
        if self.unpacked is not None:
            x.unpacked = _ptr(self.unpacked)
            x.ld_unpacked = _lmat(self.unpacked, torch.float32, "unpacked", L, n, m)
        if self.src is not None:
            x.src = self.src.as_c()
        if self.sel_sq is not None:
            _vec(self.sel_sq, torch.float32, "sel_sq", self.k)
            x.sel_sq = _ptr(self.sel_sq)
        if self.acc_sq is not None:
            _vec(self.acc_sq, torch.float32, "acc_sq", m - self.k)
            x.acc_sq = _ptr(self.acc_sq)
        if self.weight_cols is not None:
            r, c = _stored(L, n, m - self.k)
            x.weight_cols = _ptr(self.weight_cols)
            x.ld_weight_cols = _mat(self.weight_cols, torch.bfloat16, "weight_cols", r, c,
                                    device_ok=True)
        if self.acc_first is not None:
            x.acc_first = _ptr(self.acc_first)
            x.ld_acc_first = _lmat(self.acc_first, torch.bfloat16, "acc_first", L, n, m)
        return x


ZEN_TOTALS_BYTES = ctypes.sizeof(ZfZenTotals)
ZEN_STATE_BYTES = 8  # zf_zen_state: int32 length, int32 ended


def _check_dev_bytes(t: torch.Tensor, nbytes: int, name: str) -> None:
    if (t.device.type != "cuda" or not t.is_contiguous()
            or t.numel() * t.element_size() < nbytes):
        raise ValueError(f"{name}: expected a contiguous GPU tensor of at least {nbytes} bytes")


@dataclass(frozen=True)
class ZenTotals:
    """Set-wide Zen-auto totals of one step (zf_zen_totals)."""
    sum_sel: float
    sum_acc: float
    k_total: int
    u_total: int
    trigger: bool

    @staticmethod
    def from_bytes(raw: bytes) -> "ZenTotals":
        t = ZfZenTotals.from_buffer_copy(bytes(raw[:ZEN_TOTALS_BYTES]))
        return ZenTotals(t.sum_sel, t.sum_acc, t.k_total, t.u_total, bool(t.trigger))


class Plan:
    """A batch of matrices run by one launch per kernel (zf_plan_*).

    The plan's device tables and workspace live in a torch buffer owned by
    this object (sized by zf_plan_query).  The tables are uploaded on
    `stream` (default: the current stream), which is then synchronised, so
    the plan can be launched on any stream.  close() synchronises the
    device before the buffer is released (kernels in flight may still read
    the tables)."""

    def __init__(self, mats: Sequence[MatrixBuffers], stream=None):
        self.mats: List[MatrixBuffers] = list(mats)  # keeps the tensors alive
        arr = (ZfMatrix * len(self.mats))(*[b.as_c() for b in self.mats])
        nbytes = c_sz()
        _check("zf_plan_query", LIB.zf_plan_query(arr, len(self.mats), ctypes.byref(nbytes)))
        dev = self.mats[0].grad.device if self.mats[0].grad is not None else None
        if dev is None or dev.type != "cuda":
            dev = torch.device("cuda", torch.cuda.current_device())
        self.device = dev
        # 256-byte aligned start inside the buffer
        self._mem = torch.empty(nbytes.value + 256, dtype=torch.uint8, device=dev)
        base = self._mem.data_ptr()
        aligned = (base + 255) & ~255
        st = stream if stream is not None else torch.cuda.current_stream(dev)
        h = c_vp()
        _check("zf_plan_create", LIB.zf_plan_create(arr, len(self.mats), aligned, nbytes.value,
                                                   st.cuda_stream, ctypes.byref(h)))
        self._h = h
        st.synchronize()

    @property
    def device_bytes(self) -> int:
        return LIB.zf_plan_device_bytes(self._h)

    def colnorm(self, stream=None) -> None:
        _check("zf_plan_colnorm", LIB.zf_plan_colnorm(self._h, _stream(stream)))

    def colnorm_stage(self, stream=None) -> None:
        """Scores plus every channel's gradient row copied to its row of the
        bf16 first-step stage (zf_plan_colnorm_stage)."""
        _check("zf_plan_colnorm_stage", LIB.zf_plan_colnorm_stage(self._h, _stream(stream)))

    def colnorm_handover(self, scale: float, stream=None) -> None:
        """Scores plus scale x every channel's widened gradient row in its
        row of `unpacked` (zf_plan_colnorm_handover)."""
        _check("zf_plan_colnorm_handover",
               LIB.zf_plan_colnorm_handover(self._h, float(scale), _stream(stream)))

    def update_adam_handover(self, hp: AdamHparams, step: int, mode: int, stream=None) -> None:
        """Adam on the selected channels and +0.0 in their hand-over rows
        (zf_plan_update_adam_handover), after colnorm_handover."""
        c_hp = hp.as_c()
        _check("zf_plan_update_adam_handover", LIB.zf_plan_update_adam_handover(
            self._h, ctypes.byref(c_hp), step, mode, _stream(stream)))

    def topk_select(self, stream=None) -> None:
        _check("zf_plan_topk_select", LIB.zf_plan_topk_select(self._h, _stream(stream)))

    def update(self, hp: AdamHparams, step: int, mode: int, step_in_interval: int,
               accum_interval: int, adam: bool = True, pack: bool = True, stream=None) -> None:
        c_hp = hp.as_c()
        _check("zf_plan_update", LIB.zf_plan_update(
            self._h, ctypes.byref(c_hp), step, mode, step_in_interval, accum_interval,
            int(adam), int(pack), _stream(stream)))

    def unpack(self, scale: float, stream=None) -> None:
        _check("zf_plan_unpack", LIB.zf_plan_unpack(self._h, float(scale), _stream(stream)))

    def unpack_first(self, scale: float, stream=None) -> None:
        """The hand-over of a one-step interval from the bf16 stage
        (zf_plan_unpack_first)."""
        _check("zf_plan_unpack_first",
               LIB.zf_plan_unpack_first(self._h, float(scale), _stream(stream)))

    def update_handover(self, hp: AdamHparams, step: int, mode: int, step_in_interval: int,
                        accum_interval: int, scale: float, stream=None) -> None:
        """The last step of an interval with the hand-over fused in
        (zf_plan_update_handover): every matrix's `unpacked` buffer receives
        scale * the final sums; the packed buffers are only read."""
        c_hp = hp.as_c()
        _check("zf_plan_update_handover", LIB.zf_plan_update_handover(
            self._h, ctypes.byref(c_hp), step, mode, step_in_interval, accum_interval,
            float(scale), _stream(stream)))

    def update_handover_deferred(self, hp: AdamHparams, step: int, earlier: Sequence["Plan"],
                                 scale: float, stream=None) -> None:
        """The last step of an interval with deferred packing
        (zf_plan_update_handover_deferred): Adam on the selected channels and
        the hand-over of scale x the sum, in step order, of the gradients of
        the plans `earlier` (the interval's earlier steps) and this plan's."""
        hs = (c_vp * len(earlier))(*[e._h.value for e in earlier])
        c_hp = hp.as_c()
        _check("zf_plan_update_handover_deferred", LIB.zf_plan_update_handover_deferred(
            self._h, ctypes.byref(c_hp), step, hs, len(earlier), float(scale), _stream(stream)))

    def scatter_weights(self, stream=None) -> None:
        """W[:, unsel] = weight_cols of every matrix (zf_plan_scatter_weights)."""
        _check("zf_plan_scatter_weights", LIB.zf_plan_scatter_weights(self._h, _stream(stream)))

    def update_pending(self, hp: AdamHparams, step: int, accum_interval: int, pend_step: int,
                       pend_scale: float, stream=None) -> None:
        """The refresh step of the offloaded optimizer while the host still
        applies the previous interval's deferred update
        (zf_plan_update_pending): a remap + fused update against the store
        in which every column entering the selection first takes the owed
        step (pend_scale x its sums in src.pend_acc, constants of
        pend_step)."""
        c_hp = hp.as_c()
        _check("zf_plan_update_pending", LIB.zf_plan_update_pending(
            self._h, ctypes.byref(c_hp), step, accum_interval, pend_step, float(pend_scale),
            _stream(stream)))

    def scatter_weights_skip_prev(self, stream=None) -> None:
        """scatter_weights, leaving the columns of each matrix's src.prev
        selection untouched (zf_plan_scatter_weights_skip_prev)."""
        _check("zf_plan_scatter_weights_skip_prev",
               LIB.zf_plan_scatter_weights_skip_prev(self._h, _stream(stream)))

    def update_zen(self, hp: AdamHparams, step: int, mode: int, step_in_interval: int,
                   accum_interval: int, tau: float, totals: torch.Tensor, stream=None) -> None:
        """Fused update plus the Zen-auto statistics of every matrix (its
        sel_sq / acc_sq) and the set-wide totals, written to `totals` (a
        device tensor of ZEN_TOTALS_BYTES bytes, see ZenTotals)."""
        if (totals.device.type != "cuda" or not totals.is_contiguous()
                or totals.numel() * totals.element_size() < ZEN_TOTALS_BYTES):
            raise ValueError(f"totals: expected a contiguous GPU tensor of at least "
                             f"{ZEN_TOTALS_BYTES} bytes")
        c_hp = hp.as_c()
        _check("zf_plan_update_zen", LIB.zf_plan_update_zen(
            self._h, ctypes.byref(c_hp), step, mode, step_in_interval, accum_interval,
            float(tau), totals.data_ptr(), _stream(stream)))

    def update_zen_device(self, hp: AdamHparams, step: int, mode: int, accum_interval: int,
                          force_end: int, tau: float, totals: torch.Tensor,
                          state: torch.Tensor, stream=None) -> None:
        """update_zen with the interval's position read from, and the end
        decision written to, the device interval state `state` (a GPU tensor
        of ZEN_STATE_BYTES bytes; zf_plan_update_zen_device).  force_end: 0,
        1 (the caller ends the interval; handover_zen hands over) or 2
        (channel-major: the update writes the hand-over itself)."""
        _check_dev_bytes(totals, ZEN_TOTALS_BYTES, "totals")
        _check_dev_bytes(state, ZEN_STATE_BYTES, "state")
        c_hp = hp.as_c()
        _check("zf_plan_update_zen_device", LIB.zf_plan_update_zen_device(
            self._h, ctypes.byref(c_hp), step, mode, accum_interval, int(force_end),
            float(tau), totals.data_ptr(), state.data_ptr(), _stream(stream)))

    def handover_zen(self, state: torch.Tensor, stream=None) -> None:
        """The hand-over of the step update_zen_device ran, if the device
        ended the interval (zf_plan_handover_zen)."""
        _check_dev_bytes(state, ZEN_STATE_BYTES, "state")
        _check("zf_plan_handover_zen", LIB.zf_plan_handover_zen(self._h, state.data_ptr(),
                                                                _stream(stream)))

    def update_zen_deferred(self, hp: AdamHparams, step: int, mode: int, accum_interval: int,
                            earlier: Sequence["Plan"], force_end: int, tau: float,
                            totals: torch.Tensor, state: torch.Tensor, stream=None) -> None:
        """update_zen_device with deferred packing (channel-major;
        zf_plan_update_zen_deferred): the unselected channels' statistics
        are taken on the interval's running sum, summed from the gradients of
        the last position - 1 plans of `earlier` (the steps before this one,
        oldest first) and this plan's; nothing is packed.  force_end 2
        writes the hand-over."""
        _check_dev_bytes(totals, ZEN_TOTALS_BYTES, "totals")
        _check_dev_bytes(state, ZEN_STATE_BYTES, "state")
        hs = (c_vp * max(1, len(earlier)))(*[e._h.value for e in earlier])
        c_hp = hp.as_c()
        _check("zf_plan_update_zen_deferred", LIB.zf_plan_update_zen_deferred(
            self._h, ctypes.byref(c_hp), step, mode, accum_interval, hs, len(earlier),
            int(force_end), float(tau), totals.data_ptr(), state.data_ptr(), _stream(stream)))

    def handover_zen_deferred(self, earlier: Sequence["Plan"], state: torch.Tensor,
                              stream=None) -> None:
        """The hand-over of the step update_zen_deferred ran, if the device
        ended the interval (zf_plan_handover_zen_deferred)."""
        _check_dev_bytes(state, ZEN_STATE_BYTES, "state")
        hs = (c_vp * max(1, len(earlier)))(*[e._h.value for e in earlier])
        _check("zf_plan_handover_zen_deferred", LIB.zf_plan_handover_zen_deferred(
            self._h, hs, len(earlier), state.data_ptr(), _stream(stream)))

    def update_zen_pending(self, hp: AdamHparams, step: int, accum_interval: int,
                           pend_step: int, pend_scale: float, tau: float,
                           totals: torch.Tensor, stream=None) -> None:
        """update_zen for the refresh step that takes over the owed deferred
        update (zf_plan_update_zen_pending; see update_pending)."""
        if (totals.device.type != "cuda" or not totals.is_contiguous()
                or totals.numel() * totals.element_size() < ZEN_TOTALS_BYTES):
            raise ValueError(f"totals: expected a contiguous GPU tensor of at least "
                             f"{ZEN_TOTALS_BYTES} bytes")
        c_hp = hp.as_c()
        _check("zf_plan_update_zen_pending", LIB.zf_plan_update_zen_pending(
            self._h, ctypes.byref(c_hp), step, accum_interval, pend_step, float(pend_scale),
            float(tau), totals.data_ptr(), _stream(stream)))

    def close(self) -> None:
        if getattr(self, "_h", None):
            torch.cuda.synchronize(self.device)  # launches may still read the tables
            LIB.zf_plan_destroy(self._h)
            self._h = None
            self._mem = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
