"""Second, bit-level numpy oracle -- TEST INFRASTRUCTURE ONLY.

Same definitions as ref.c, written independently so the two can be checked
against each other bit for bit:

* widening bf16 -> fp32 places the 16 bits in the high half of a 32-bit word;
* fp32 -> bf16 round-to-nearest-even adds 0x7FFF plus the kept LSB to the
  32-bit pattern and keeps the high half (carries into the exponent give the
  next binade and, past the largest finite value, infinity);
* the reduction adds rank after rank in ascending order in numpy float32
  (the one-shot pull-and-reduce loop of Sec. 4.2);
* the epilogue (paper silent) is evaluated in float64, with a vectorised
  round-half-even to bf16 done by scaling to the bf16 grid and ``np.rint``.
"""
from __future__ import annotations

import numpy as np


def widen(b: np.ndarray) -> np.ndarray:
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def narrow_rne_f32(f: np.ndarray) -> np.ndarray:
    f = np.asarray(f, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    r = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    nan = np.isnan(f)
    r = np.where(nan, (u >> 16) | 0x40, r)
    return r.astype(np.uint16)


def reduce(x: np.ndarray) -> np.ndarray:
    x = np.asarray(x, dtype=np.uint16)
    acc = widen(x[0]).copy()
    with np.errstate(over="ignore", invalid="ignore"):
        for r in range(1, x.shape[0]):
            acc = (acc + widen(x[r])).astype(np.float32)
    return narrow_rne_f32(acc)


def narrow_rne_f64(v: np.ndarray) -> np.ndarray:
    """float64 -> bf16 bits, one rounding, ties to even."""
    v = np.asarray(v, dtype=np.float64)
    sign = np.signbit(v)
    a = np.abs(v)
    with np.errstate(divide="ignore", invalid="ignore", over="ignore"):
        _, e2 = np.frexp(a)
        ulp_exp = np.maximum(e2 - 8, -133)
        q = np.rint(np.ldexp(a, -ulp_exp))
        r = np.ldexp(q, ulp_exp)
    r = np.where(r >= 2.0 ** 128, np.inf, r)
    # r is now exactly a bf16 value (or inf): its float32 pattern's high half.
    bits = (r.astype(np.float32).view(np.uint32) >> 16).astype(np.uint16)
    bits = np.where(np.isnan(v), np.uint16(0x7FC0), bits)
    return np.where(sign, bits | np.uint16(0x8000), bits).astype(np.uint16)


def residual_rmsnorm(a, res, w, eps):
    a64 = widen(a).astype(np.float64)
    r64 = widen(res).astype(np.float64)
    res2 = narrow_rne_f64(a64 + r64)
    v = widen(res2).astype(np.float64)
    T, H = v.shape
    ss = np.zeros(T)
    for h in range(H):  # ascending h, as the C oracle
        ss = ss + v[:, h] * v[:, h]
    inv = 1.0 / np.sqrt(ss / H + eps)
    y = narrow_rne_f64(v * inv[:, None] * widen(w).astype(np.float64)[None, :])
    return res2, y
