"""Pins of the oracle's RETAIN-LOW quantiser (int4, fp16 scale per 32
elements; the paper names no low-bit format, Section 3.1 only orders the
actions by memory cost)."""

import numpy as np
import pytest
import torch

import oracle
from tests import pins


def bf16_bits(x) -> np.ndarray:
    t = torch.as_tensor(x, dtype=torch.float32).to(torch.bfloat16)
    return t.view(torch.int16).numpy().astype(np.int64) & 0xFFFF


def test_scale_exhaustive_vs_numpy():
    a = pins.all_nonneg_finite_bf16()
    assert a.size == 32640
    assert pins.scale_mismatches_numpy(oracle.fp16_scale_bits, a) == 0


def test_scale_exhaustive_vs_fraction():
    a = pins.all_nonneg_finite_bf16()
    assert pins.scale_mismatches_fraction(oracle.fp16_scale_bits, a) == 0


def _groups(rng, n):
    """Random groups spanning the interesting ranges: normal data, wide
    exponents, outliers, subnormals, huge values, exact ties, all-equal."""
    out = []
    k = n // 6
    out.append(rng.standard_normal((k, 32)))
    out.append(rng.standard_normal((k, 32)) * np.exp2(rng.integers(-140, 120, size=(k, 1))))
    g = rng.standard_normal((k, 32))
    g[:, rng.integers(0, 32)] *= 64
    out.append(g)
    out.append(rng.standard_normal((k, 32)) * 2.0 ** -130)               # bf16 subnormals
    out.append(rng.standard_normal((k, 32)) * 1e37)                      # scale saturation
    s = np.exp2(rng.integers(-20, 10, size=(k, 1)).astype(np.float64))
    h = rng.integers(-7, 7, size=(k, 32)) + 0.5                          # exact half-integers
    t = h * s
    t[:, 0] = 7 * s[:, 0]                                                # absmax 7s -> scale s
    out.append(t)
    x = np.concatenate(out)
    return bf16_bits(x.astype(np.float32))


def test_codes_vs_fraction_bruteforce():
    rng = np.random.default_rng(7)
    x = _groups(rng, 3000)
    assert pins.codes_mismatches_fraction(oracle.quantize_groups, x) == 0


def test_codes_vs_float_rint_many():
    rng = np.random.default_rng(8)
    x = _groups(rng, 600000)
    assert pins.codes_mismatches_float(oracle.quantize_groups, x) == 0


def test_ties_round_to_even():
    # absmax 7 gives s = 1 exactly; x/s = 2.5, 3.5, -2.5, 0.5, 1.5, -0.5 are ties.
    x = bf16_bits([7.0, 2.5, 3.5, -2.5, 0.5, 1.5, -0.5, 4.5, 5.5, 6.5] + [0.0] * 22)
    codes, s = oracle.quantize_groups(x[None])
    assert int(s[0, 0]) == 0x3C00
    assert codes[0, :10].tolist() == [7, 2, 4, -2, 0, 2, 0, 4, 6, 6]


def test_special_groups():
    zero = bf16_bits([0.0] * 32)
    c, s = oracle.quantize_groups(zero[None])
    assert int(s[0, 0]) == 0 and not c.any()
    negzero = bf16_bits([-0.0] * 32)
    c, s = oracle.quantize_groups(negzero[None])
    assert int(s[0, 0]) == 0 and not c.any()
    eq = bf16_bits([3.0] * 32)
    c, s = oracle.quantize_groups(eq[None])
    assert (c == 7).all()
    neq = bf16_bits([-3.0] * 32)
    c, s = oracle.quantize_groups(neq[None])
    assert (c == -7).all()
    huge = bf16_bits([3e38] + [1e30] * 31)
    c, s = oracle.quantize_groups(huge[None])
    assert int(s[0, 0]) == 0x7BFF and c[0, 0] == 7 and (c[0, 1:] == 7).all()


def test_invariants_on_random_groups():
    rng = np.random.default_rng(9)
    x = _groups(rng, 60000)
    codes, sbits = oracle.quantize_groups(x)
    assert np.abs(codes.astype(np.int64)).max() <= 7
    xf = oracle.bf16_to_f64(x)
    s = oracle.fp16_to_f64(sbits).reshape(-1)
    amax_idx = np.abs(xf).argmax(axis=1)
    sat = sbits.reshape(-1) == 0x7BFF
    nz = s > 0
    # The absmax element maps to +-7 whenever the scale is a normal fp16 number
    # (below 2**-14 the fp16 grid is too coarse for absmax/7 to land near 7s).
    am = np.abs(codes[np.arange(x.shape[0]), amax_idx].astype(np.int64))
    assert (am[s >= 2.0 ** -14] == 7).all()
    # Reconstruction error at most s/2 where nothing was clamped.
    xhat = oracle.dequant(codes, sbits)
    clamped = (np.abs(xf) > 7.5 * s[:, None]).any(axis=1) | sat
    ok = nz & ~clamped
    err = np.abs(xf - xhat)[ok].max(axis=1)
    assert (err <= s[ok] / 2).all()


def test_pack_nibble_order_literal():
    # Element 2j in the low nibble of byte j, two's complement.
    codes = np.array([1, -1, 7, -7, 0, 3, -8 + 1, 2], dtype=np.int8)
    packed = oracle.pack_nibbles(codes)
    assert packed.tolist() == [0xF1, 0x97, 0x30, 0x29]
    assert oracle.unpack_nibbles(packed).tolist() == codes.tolist()


def test_pack_roundtrip_random():
    rng = np.random.default_rng(3)
    c = rng.integers(-7, 8, size=(100, 64)).astype(np.int8)
    assert (oracle.unpack_nibbles(oracle.pack_nibbles(c)) == c).all()


def test_dequant_exact():
    # q * s is exact: 4-bit times 11-bit significands.
    codes = np.array([[7, -7, 1, -1] + [0] * 28], dtype=np.int8)
    sb = np.array([[0x3092]], dtype=np.uint16)
    s = float(np.array([0x3092], dtype=np.uint16).view(np.float16)[0])
    got = oracle.dequant(codes, sb)[0, :4]
    assert got.tolist() == [7 * s, -7 * s, s, -s]


@pytest.mark.parametrize("mutant", ["half_up", "exponent_off_by_one", "sign_dropped"])
def test_planted_quantiser_mistakes_are_caught(mutant, monkeypatch):
    """A plausible slip inside the oracle's quantiser fails a pin."""
    import oracle.pask_oracle as po

    if mutant == "half_up":                       # ties rounded up instead of to even
        def bad(num, den):
            q, r = np.divmod(num, den)
            return q + (2 * r >= den).astype(np.int64)
        monkeypatch.setattr(po, "_rne_div", bad)
    elif mutant == "exponent_off_by_one":         # binade of absmax/7 misjudged
        good = po._floor_log2_ratio
        monkeypatch.setattr(po, "_floor_log2_ratio", lambda m, e, d: good(m, e, d) + 1)
    else:                                         # magnitude quantised, sign lost
        good_mag = po.bf16_mag

        def bad_mag(bits):
            s, m, e = good_mag(bits)
            return np.zeros_like(s), m, e
        monkeypatch.setattr(po, "bf16_mag", bad_mag)
    a = pins.all_nonneg_finite_bf16()
    x = _groups(np.random.default_rng(1), 6000)
    caught = (pins.scale_mismatches_numpy(po.fp16_scale_bits, a) > 0
              or pins.codes_mismatches_float(po.quantize_groups, x) > 0)
    assert caught


def test_planted_nibble_swap_is_caught():
    def swapped(codes):
        c = np.asarray(codes, dtype=np.int64) & 0xF
        return (c[..., 1::2] | (c[..., 0::2] << 4)).astype(np.uint8)
    codes = np.array([1, -1, 7, -7, 0, 3, -8 + 1, 2], dtype=np.int8)
    assert swapped(codes).tolist() != [0xF1, 0x97, 0x30, 0x29]
