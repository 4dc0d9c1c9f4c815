"""Seeded generators for synthetic Llama-shaped gradients.

What is drawn (all seeded, all reproducible on the device they are drawn on):

* Per-column scales s_j = exp(sigma * z_j), z_j ~ N(0, 1): heavy-tailed
  channel energy, standing in for the paper's observation that a small share
  of gradients carries most of the gradient norm (Problems and Insights,
  Insight #1) and that it concentrates on input channels (Insight #2).
* Temporal jitter s_{j,t} = s_j * exp(rel * xi_{j,t}) around a persistent
  base, standing in for the temporal locality of important channels.
* Gradient G[i, j] = bf16(sign_ij * b[(i + c_j) mod n] * s_j), where b ~
  N(0, 1)^n is one draw per matrix and step, c_j a random cyclic offset and
  sign_ij a random sign.  Every column is a signed, shifted copy of the same
  N(0, 1) sample, so each element is marginally N(0, 1) * s_j and every
  column carries the same noise energy sum(b^2).  Column energies are
  therefore proportional to s_j^2 up to bf16 rounding, which lets the
  generator space them by acting on the scales alone: it never computes a
  norm of G.
* Master weights N(0, std^2) in fp32, bf16 weights = their bf16 rounding
  (torch's cast).
* `gradient_iid`: the same scales with every element its own N(0, 1) draw,
  for tests of selection on columns whose noise energies differ.

Nothing here computes column norms, selections, optimizer steps or packed
buffers.
"""

from __future__ import annotations

import hashlib
import math
from typing import Optional

import numpy as np
import torch

from .configs import Workload

# Relative gap imposed on column scales where spacing is requested.  Column
# energies scale with s^2, so a 1.5e-3 gap in s gives ~3e-3 in energy, which
# leaves a margin over bf16 rounding (a few 1e-4 at n = 4096) for the
# realised squared norms to differ by more than 1e-3.
DEFAULT_SCALE_GAP = 1.5e-3

# Row chunk used when drawing large gradients (bounds temporaries; fixed so
# that draws are reproducible).
_CHUNK_ROWS = 2048


def derive_seed(*parts) -> int:
    """Deterministic 63-bit seed from a tuple of ints/strings."""
    h = hashlib.blake2b(repr(tuple(parts)).encode(), digest_size=8).digest()
    return int.from_bytes(h, "little") & ((1 << 63) - 1)


def _gen(seed: int, device) -> torch.Generator:
    g = torch.Generator(device=torch.device(device))
    g.manual_seed(int(seed))
    return g


def base_scales(m: int, sigma: float, seed: int) -> torch.Tensor:
    """Lognormal(0, sigma) per-column scales, float64 on the CPU."""
    g = _gen(seed, "cpu")
    z = torch.randn(m, generator=g, dtype=torch.float64)
    return torch.exp(sigma * z)


def jittered_scales(base: torch.Tensor, rel: float, seed: int) -> torch.Tensor:
    """base * exp(rel * xi), xi ~ N(0, 1): jitter around a persistent base."""
    if rel == 0.0:
        return base.clone()
    g = _gen(seed, "cpu")
    xi = torch.randn(base.numel(), generator=g, dtype=torch.float64)
    return base * torch.exp(rel * xi)


def space_all_pairs(scales: torch.Tensor, gap: float = DEFAULT_SCALE_GAP) -> torch.Tensor:
    """Stretch scales so that every pair of sorted neighbours differs by a
    factor of at least (1 + gap).  Works in the log domain:
    l'_r = max(l_r, l'_{r-1} + log1p(gap)) over the ascending order."""
    s = scales.detach().cpu().numpy().astype(np.float64)
    m = s.size
    if m < 2:
        return scales.clone()
    order = np.argsort(s, kind="stable")
    ls = np.log(s[order])
    delta = math.log1p(gap) * (1.0 + 1e-9)
    r = np.arange(m, dtype=np.float64) * delta
    ls = np.maximum.accumulate(ls - r) + r
    out = np.empty_like(s)
    out[order] = np.exp(ls)
    return torch.from_numpy(out)


def space_boundary(scales: torch.Tensor, k: int, gap: float = DEFAULT_SCALE_GAP) -> torch.Tensor:
    """Make the k-th largest scale exceed the (k+1)-th by a factor of at least
    (1 + gap), by multiplying the k largest scales by one common factor (their
    internal order is kept)."""
    s = scales.detach().cpu().numpy().astype(np.float64).copy()
    m = s.size
    if k <= 0 or k >= m:
        return torch.from_numpy(s)
    order = np.argsort(-s, kind="stable")
    kth, nxt = s[order[k - 1]], s[order[k]]
    want = nxt * (1.0 + gap) * (1.0 + 1e-9)
    if kth < want:
        s[order[:k]] *= want / kth
    return torch.from_numpy(s)


def step_scales(wl: Workload, q: int, t: int, k_boundary: Optional[int] = None,
                gap: float = DEFAULT_SCALE_GAP) -> torch.Tensor:
    """Column scales of matrix q of workload wl at 1-based step t (float64, CPU).

    k_boundary is the number of columns the caller will select; it is only
    used for the "boundary" spacing rule."""
    mt = wl.matrices[q]
    base = base_scales(mt.m, wl.sigma, derive_seed(wl.seed, q, "base"))
    s = jittered_scales(base, wl.jitter, derive_seed(wl.seed, q, "jitter", t))
    if wl.spacing == "all":
        s = space_all_pairs(s, gap)
    elif wl.spacing == "boundary":
        if k_boundary is not None:
            s = space_boundary(s, k_boundary, gap)
    elif wl.spacing != "none":
        raise ValueError(f"unknown spacing rule {wl.spacing!r}")
    return s


def gradient(n: int, m: int, scales: torch.Tensor, seed: int,
             device="cpu", out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """bf16 gradient [n, m]: sign * b[(i + c_j) mod n] * s_j, rounded by torch's
    fp32 -> bf16 cast.  `out` may be a preallocated (possibly row-strided)
    [n, m] bf16 view on `device`."""
    device = torch.device(device)
    if out is None:
        out = torch.empty(n, m, dtype=torch.bfloat16, device=device)
    if n == 0 or m == 0:
        return out
    g = _gen(seed, device)
    b = torch.randn(n, generator=g, device=device, dtype=torch.float32)
    c = torch.randint(0, n, (m,), generator=g, device=device, dtype=torch.int64)
    s32 = scales.to(torch.float32).to(device)
    rows = torch.arange(n, device=device, dtype=torch.int64)
    for r0 in range(0, n, _CHUNK_ROWS):
        r1 = min(n, r0 + _CHUNK_ROWS)
        idx = torch.remainder(rows[r0:r1, None] + c[None, :], n)
        sign = torch.randint(0, 2, (r1 - r0, m), generator=g, device=device,
                             dtype=torch.int8)
        z = b[idx]
        z = torch.where(sign.bool(), -z, z)
        out[r0:r1] = (z * s32[None, :]).to(torch.bfloat16)
    return out


def gradient_iid(n: int, m: int, scales: torch.Tensor, seed: int,
                 device="cpu") -> torch.Tensor:
    """bf16 gradient [n, m] with independent elements: bf16(z_ij * s_j), z_ij ~
    N(0, 1) each its own draw (torch's CPU generator, then moved to
    `device`, so that the same seed gives the same bits wherever the test
    runs).  Unlike `gradient`, each column carries its own noise energy, so
    column energies only approximately follow s_j^2 and no spacing can be
    imposed through the scales."""
    out = torch.empty(n, m, dtype=torch.bfloat16)
    if n > 0 and m > 0:
        g = _gen(seed, "cpu")
        s32 = scales.to(torch.float32).cpu()
        for r0 in range(0, n, _CHUNK_ROWS):
            r1 = min(n, r0 + _CHUNK_ROWS)
            z = torch.randn(r1 - r0, m, generator=g, dtype=torch.float32)
            out[r0:r1] = (z * s32[None, :]).to(torch.bfloat16)
    return out.to(torch.device(device))


def master_weights(n: int, m: int, seed: int, std: float = 0.02,
                   device="cpu") -> torch.Tensor:
    """fp32 master weights N(0, std^2), [n, m]."""
    g = _gen(seed, device)
    w = torch.randn(n, m, generator=g, device=torch.device(device), dtype=torch.float32)
    return w * torch.tensor(std, dtype=torch.float32, device=w.device)


def score_vector(m: int, seed: int, kind: str = "lognormal") -> torch.Tensor:
    """Stand-alone fp32 score vectors for exercising selection in isolation."""
    g = _gen(seed, "cpu")
    if kind == "lognormal":
        return torch.exp(1.5 * torch.randn(m, generator=g, dtype=torch.float64)).to(torch.float32)
    if kind == "wide":
        # Spans most fp32 exponents, including subnormals and very large values.
        e = torch.randint(-149, 127, (m,), generator=g, dtype=torch.int64).to(torch.float64)
        f = 1.0 + torch.rand(m, generator=g, dtype=torch.float64)
        return (f * torch.pow(2.0, e)).to(torch.float32)
    if kind == "ties":
        return torch.randint(0, 4, (m,), generator=g, dtype=torch.int64).to(torch.float32)
    if kind == "few-distinct":
        vals = torch.tensor([0.0, 1.5, 1e-3, 7.0, 3.25e5], dtype=torch.float32)
        return vals[torch.randint(0, vals.numel(), (m,), generator=g)]
    if kind == "zeros":
        return torch.zeros(m, dtype=torch.float32)
    if kind == "constant":
        return torch.full((m,), 2.5, dtype=torch.float32)
    if kind == "signed-zero":
        v = torch.randint(0, 3, (m,), generator=g, dtype=torch.int64)
        out = torch.where(v == 0, torch.tensor(0.0), torch.where(v == 1, torch.tensor(-0.0),
                          torch.tensor(1.0)))
        return out.to(torch.float32)
    raise ValueError(f"unknown score vector kind {kind!r}")
