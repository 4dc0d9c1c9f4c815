"""Seeded bit-pattern generators for the numerical edge cases of the optimizer
step: bf16 gradients and fp32 states and sums spread over the whole exponent
range of their formats.

Every value is drawn as a bit pattern (sign, exponent field, mantissa), by
class:

  zero     +0.0 and -0.0
  eps      |x| in about [1e-9, 1e-7], where Adam's eps (1e-8) decides the
           denominator
  tiny     |x| < 2^-64 (bf16 and fp32 subnormals included): the squares of
           such values are subnormal in fp32 or underflow to zero
  huge     |x| >= 2^64: their squares overflow fp32
  any      any finite pattern
  typical  |x| within a few binades of 1e-3 .. 1

Nothing here computes an optimizer step, a norm or a rounding: both the
oracle side of a test and the HIP path consume the patterns as they are.
"""

from __future__ import annotations

import numpy as np

from .synth import derive_seed

# exponent fields (bf16 and fp32 share the 8-bit field, bias 127)
_EXP = {
    "eps": (97, 103),       # 2^-30 .. 2^-24 (about 9.3e-10 .. 1.2e-7)
    "tiny": (0, 62),        # subnormal (field 0) .. below 2^-64
    "huge": (191, 254),     # 2^64 .. the largest finite binade
    "any": (0, 254),
    "typical": (117, 127),  # 2^-10 .. 2^0
}
GRAD_CLASSES = ("zero", "eps", "tiny", "huge", "any", "typical")


def _patterns(shape, seed, classes, mant_bits, sign=True):
    """uint32 patterns with an 8-bit exponent field above `mant_bits`
    mantissa bits; each element takes a class drawn uniformly."""
    rng = np.random.default_rng(seed)
    cls = rng.integers(0, len(classes), size=shape)
    e = np.zeros(shape, np.uint32)
    for c, name in enumerate(classes):
        sel = cls == c
        if name == "zero":
            continue
        lo, hi = _EXP[name]
        e[sel] = rng.integers(lo, hi + 1, size=int(sel.sum()), dtype=np.uint32)
        if name == "tiny":  # a quarter of them subnormal
            sub = sel & (rng.random(shape) < 0.25)
            e[sub] = 0
    mant = rng.integers(0, 1 << mant_bits, size=shape, dtype=np.uint32)
    zero = np.isin(cls, [classes.index("zero")]) if "zero" in classes else np.zeros(shape, bool)
    mant[zero] = 0
    # a subnormal pattern needs a nonzero mantissa to be one (else it is a zero)
    sub = (e == 0) & ~zero
    mant[sub] |= 1
    s = (rng.integers(0, 2, size=shape, dtype=np.uint32) if sign
         else np.zeros(shape, np.uint32))
    return (s << np.uint32(31)) | (e << np.uint32(23)) | (mant << np.uint32(23 - mant_bits))


def edge_bf16(shape, seed) -> np.ndarray:
    """bf16 bit patterns (uint16) over every class above."""
    p = _patterns(shape, derive_seed("edge-bf16", seed), GRAD_CLASSES, 7)
    return (p >> np.uint32(16)).astype(np.uint16)


def edge_f32(shape, seed, kind: str) -> np.ndarray:
    """fp32 values of an optimizer buffer over the classes that buffer can
    hold.  kind: "master" (signed; also bf16 rounding ties and near-ties,
    low halves 0x8000, 0x7fff, 0x8001), "first" (signed first moments),
    "second" (second moments: >= +0, -0.0 included), "sum" (signed packed
    sums, the gradient's classes at fp32 precision)."""
    if kind not in ("master", "first", "second", "sum"):
        raise ValueError(f"unknown kind {kind!r}")
    classes = {"master": ("zero", "tiny", "typical", "huge", "any"),
               "first": ("zero", "eps", "tiny", "typical", "huge"),
               "second": ("zero", "eps", "tiny", "typical", "huge"),
               "sum": GRAD_CLASSES}[kind]
    seed = derive_seed("edge-f32", kind, seed)
    p = _patterns(shape, seed, classes, 23, sign=kind != "second")
    if kind == "second":
        rng = np.random.default_rng(seed + 1)
        neg0 = rng.random(shape) < 0.02
        p[neg0] = np.uint32(0x80000000)
    if kind == "master":
        rng = np.random.default_rng(seed + 2)
        tie = rng.integers(0, 4, size=shape)
        low = np.array([0, 0x8000, 0x7FFF, 0x8001], np.uint32)[tie]
        # (the exponent field stays below 255, so these stay finite)
        p = np.where(tie == 0, p, (p & np.uint32(0xFFFF0000)) | low)
    return p.view(np.float32)


def sprinkle_nonfinite(M: np.ndarray, V: np.ndarray, seed, frac: float = 0.03):
    """Copies of first / second moments with infinities at seeded positions:
    some first moments +-inf, some second moments +inf, and some elements
    with both (whose step divides infinity by infinity)."""
    rng = np.random.default_rng(derive_seed("edge-nonfinite", seed))
    M = np.array(M, np.float32, copy=True)
    V = np.array(V, np.float32, copy=True)
    r = rng.random(M.shape)
    m_inf = r < frac
    v_inf = (r >= frac / 2) & (r < 2 * frac)
    M[m_inf] = np.where(rng.random(int(m_inf.sum())) < 0.5, np.inf, -np.inf).astype(np.float32)
    V[v_inf] = np.float32(np.inf)
    return M, V
