"""Helpers shared by the GPU parity tests (conversions and comparisons)."""
import numpy as np
import torch


def dev():
    return torch.device("cuda")


def bits_np(t: torch.Tensor) -> np.ndarray:
    """bf16 tensor -> uint16 numpy bit patterns (host copy)."""
    return t.detach().contiguous().view(torch.int16).cpu().numpy().view(np.uint16)


def bf16_dev(bits: np.ndarray, ld: int = None, offset: int = 0) -> torch.Tensor:
    """uint16 bit patterns -> bf16 device tensor [n, m], optionally inside a
    wider row-major buffer (row stride ld, first column at `offset`)."""
    bits = np.ascontiguousarray(bits, dtype=np.uint16)
    n, m = bits.shape
    ld = m if ld is None else ld
    buf = torch.zeros(max(n, 1) * ld + offset + 8, dtype=torch.int16)
    if n:
        view = buf[offset: offset + n * ld].view(n, ld)[:, :m]
        view.copy_(torch.from_numpy(bits.view(np.int16)))
    dbuf = buf.to(dev()).view(torch.bfloat16)
    return dbuf[offset: offset + n * ld].view(n, ld)[:, :m] if n else dbuf[:0].view(0, m)


def f32_np(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().numpy()


def f32_dev(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(dev())


def mask_np(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().numpy().view(np.uint64)


def rel_close(got, want, rtol, floor=None):
    """|got - want| <= rtol * |want| (+ floor), zeros exact; returns (ok, worst)."""
    got = np.asarray(got, np.float64)
    want = np.asarray(want, np.float64)
    tol = rtol * np.abs(want)
    if floor is not None:
        tol = tol + floor
    err = np.abs(got - want)
    bad = err > tol
    worst = float((err / np.maximum(np.abs(want), 1e-300)).max()) if err.size else 0.0
    return (not bad.any()), worst


def same_bits(a, b) -> bool:
    """Equal shapes, element sizes and bit patterns (no byte-string copies)."""
    a = np.ascontiguousarray(a)
    b = np.ascontiguousarray(b)
    if a.shape != b.shape or a.dtype.itemsize != b.dtype.itemsize:
        return False
    return bool(np.array_equal(a.reshape(-1).view(np.uint8), b.reshape(-1).view(np.uint8)))
