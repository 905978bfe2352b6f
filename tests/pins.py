"""Independent checks that pin the oracle to something other than itself.

Each function takes the oracle-like callable under test and returns the
number of disagreements with a reference that does not reuse the oracle's
arithmetic: exact rational arithmetic (fractions.Fraction) over an enumerated
fp16 grid, numpy/torch library routines, or closed forms.  The planted-mistake
tests call them with deliberately broken copies of oracle functions to show
that a plausible slip is caught.
"""

from __future__ import annotations

import bisect
from fractions import Fraction

import numpy as np
import torch


def all_nonneg_finite_bf16() -> np.ndarray:
    """Every non-negative finite bf16 bit pattern (255 exponents x 128 mantissas, incl. 0)."""
    return np.arange(0x0000, 0x7F80, dtype=np.int64)


def bf16_fraction(bits: int) -> Fraction:
    bits &= 0xFFFF
    sign = -1 if bits >> 15 else 1
    ex, man = (bits >> 7) & 0xFF, bits & 0x7F
    if ex == 0:
        return sign * Fraction(man, 1) * Fraction(2) ** -133
    return sign * Fraction(128 + man) * Fraction(2) ** (ex - 134)


def fp16_fraction(bits: int) -> Fraction:
    ex, man = (bits >> 10) & 0x1F, bits & 0x3FF
    sign = -1 if (bits >> 15) & 1 else 1
    if ex == 0:
        return sign * Fraction(man) * Fraction(2) ** -24
    return sign * Fraction(1024 + man) * Fraction(2) ** (ex - 25)


_FP16_GRID = [fp16_fraction(b) for b in range(0, 0x7C00)]     # sorted, 0 .. 65504


def fp16_rne_fraction(r: Fraction) -> int:
    """Nearest finite non-negative fp16 to r >= 0 (ties to even mantissa),
    saturating at 65504, by search over the enumerated grid."""
    i = bisect.bisect_left(_FP16_GRID, r)
    if i >= len(_FP16_GRID):
        return 0x7BFF
    if _FP16_GRID[i] == r:
        return i
    if i == 0:
        return 0
    lo, hi = i - 1, i
    dl, dh = r - _FP16_GRID[lo], _FP16_GRID[hi] - r
    if dl < dh:
        return lo
    if dh < dl:
        return hi
    return lo if lo % 2 == 0 else hi


def rne_fraction(r: Fraction) -> int:
    """Round a rational to the nearest integer, ties to even."""
    f = r.numerator // r.denominator
    rem = r - f
    if rem > Fraction(1, 2):
        return f + 1
    if rem < Fraction(1, 2):
        return f
    return f if f % 2 == 0 else f + 1


def scale_mismatches_fraction(scale_fn, absmax_bits) -> int:
    got = np.asarray(scale_fn(np.asarray(absmax_bits)), dtype=np.int64)
    bad = 0
    for a, g in zip(absmax_bits.tolist(), got.tolist()):
        if fp16_rne_fraction(bf16_fraction(a) / 7) != g:
            bad += 1
    return bad


def scale_mismatches_numpy(scale_fn, absmax_bits) -> int:
    """numpy reference: float64 division (correctly rounded) then RNE to fp16;
    double rounding is innocuous since 53 >= 2*11 + 2."""
    a = torch.tensor(absmax_bits.astype(np.int32).astype(np.int16)).view(torch.bfloat16).double().numpy()
    r = a / 7.0
    r = np.minimum(r, 65504.0)
    ref = r.astype(np.float16).view(np.uint16).astype(np.int64)
    got = np.asarray(scale_fn(absmax_bits), dtype=np.int64)
    return int((ref != got).sum())


def codes_mismatches_fraction(quant_fn, x_bits: np.ndarray) -> int:
    """x_bits [n_groups, 32].  Reference per group: s = nearest fp16 to
    absmax/7 (saturated); q_i = clamp(RNE(x_i / s), -7, 7); q = 0 if s = 0."""
    codes, sbits = quant_fn(x_bits)
    codes = np.asarray(codes).reshape(x_bits.shape)
    sbits = np.asarray(sbits).reshape(x_bits.shape[0])
    bad = 0
    for gi in range(x_bits.shape[0]):
        vals = [bf16_fraction(int(b)) for b in x_bits[gi]]
        a = max(abs(v) for v in vals)
        sb = fp16_rne_fraction(a / 7)
        if sb != int(sbits[gi]):
            bad += 1
            continue
        s = fp16_fraction(sb)
        for j, v in enumerate(vals):
            q = 0 if s == 0 else max(-7, min(7, rne_fraction(v / s)))
            if q != int(codes[gi, j]):
                bad += 1
                break
    return bad


def codes_mismatches_float(quant_fn, x_bits: np.ndarray) -> int:
    """numpy reference for many groups: q = rint(x / s) in float64.  x/s is
    either an exact half-integer (representable, so rint sees the tie) or at
    least 2**-12 from a tie, far beyond the float64 division error."""
    codes, sbits = quant_fn(x_bits)
    x = torch.tensor(x_bits.astype(np.int32).astype(np.int16)).view(torch.bfloat16).double().numpy()
    s = np.asarray(sbits, dtype=np.uint16).view(np.float16).astype(np.float64).reshape(-1, 1)
    with np.errstate(divide="ignore", invalid="ignore"):
        q = np.where(s == 0, 0.0, np.rint(x / np.where(s == 0, 1.0, s)))
    q = np.clip(q, -7, 7).astype(np.int64)
    return int((q != np.asarray(codes, dtype=np.int64).reshape(q.shape)).any(axis=-1).sum())


def sdpa_gqa(q, k, v, scale):
    """torch scaled_dot_product_attention in fp64, KV heads repeated to the
    query heads in repeat_kv order (query head h reads KV head h // G).
    q [Hq, D], k/v [n, Hkv, D] numpy fp64 -> o [Hq, D]."""
    qt = torch.from_numpy(np.asarray(q, dtype=np.float64))[None, :, None, :]       # [1, Hq, 1, D]
    kt = torch.from_numpy(np.asarray(k, dtype=np.float64)).permute(1, 0, 2)[None]  # [1, Hkv, n, D]
    vt = torch.from_numpy(np.asarray(v, dtype=np.float64)).permute(1, 0, 2)[None]
    g = qt.shape[1] // kt.shape[1]
    kt = kt.repeat_interleave(g, dim=1)
    vt = vt.repeat_interleave(g, dim=1)
    o = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, scale=scale)
    return o[0, :, 0, :].numpy()
