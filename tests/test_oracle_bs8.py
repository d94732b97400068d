"""Pins of the oracle's block-size-8 formats (IF4-BS8, IF3-BS8, NVFP4-BS8;
Sec. 5.1 and Table 6 (App. D): one E4M3 scale per 8 values, 5.0 and 4.0 bits per
parameter for IF4-BS8 and IF3-BS8).

- Bit budget: codes + scales of a tensor come to Table 6's bits/parameter.
- Reduction to the pinned 16-value algorithm: a group of 8 quantizes exactly
  like the same 8 values followed by 8 zeros in the 16-value format (zeros
  leave max|X_g|, both candidates' errors and therefore the choice
  unchanged), for every group of a tensor, with the same alpha.
- Brute force over every code vector of tiny 8-value groups, exact
  rationals (least-squares candidates, strict "<" selection).
- Smaller blocks lose less: per-tensor MSE on N(0,1) below the 16-value
  format's, and IF4-BS8 never worse than NVFP4-BS8 group by group.
"""
import itertools
from fractions import Fraction

import numpy as np
import pytest

PAIRS = [(7, 0), (8, 2), (9, 1)]  # (block-8 format, its 16-value counterpart)


@pytest.mark.parametrize("fmt,bits_per_param", [(7, 5.0), (8, 4.0), (9, 5.0)])
def test_bits_per_parameter(oracle, fmt, bits_per_param):
    rows, cols = 32, 256
    (cr, cc), (sr, sc) = oracle.codes_shape(fmt, rows, cols)
    assert (cr * cc + sr * sc) * 8 / (rows * cols) == bits_per_param
    assert oracle.group_size(fmt) == 8


@pytest.mark.parametrize("fmt8,fmt16", PAIRS)
@pytest.mark.parametrize("flags", [0, 4])  # round to nearest; with the 16/17 margin
def test_group_of_8_is_16_with_zero_padding(oracle, fmt8, fmt16, flags):
    rng = np.random.default_rng(200 + fmt8)
    x = rng.standard_t(3, (16, 128)).astype(np.float32)
    x[:, ::13] *= 30
    xb = oracle.bf16_bits(x)
    c8, s8, a8 = oracle.quantize(xb, fmt8, flags)
    assert a8 == oracle.tensor_scale(fmt16, float(np.abs(oracle.bf16_to_f32(xb)).max()), flags)
    # each 8-value group, padded with 8 zeros, in the 16-value format
    pad = np.zeros((16, 256), dtype=np.uint16)
    xg = xb.reshape(16, 16, 8)
    pad.reshape(16, 16, 16)[:, :, :8] = xg
    c16, s16, _ = oracle.quantize(pad, fmt16, flags | oracle.SCALE_IN, tensor_scale=a8)
    np.testing.assert_array_equal(s8, s16)
    bits = oracle.BITS[fmt8]
    for r in range(16):
        for g in range(16):
            want = oracle.unpack_group(fmt16, c16[r, g * 2 * bits:(g + 1) * 2 * bits])[:8]
            got = oracle.unpack_group(fmt8, c8[r, g * bits:(g + 1) * bits])
            np.testing.assert_array_equal(got, want)


def _value(oracle, fmt, code, is_int):
    bits = oracle.BITS[fmt]
    c = int(code)
    if is_int:
        return c - (1 << bits) if c & (1 << (bits - 1)) else c
    mag = Fraction(oracle.fp_magnitude(fmt, c & ((1 << (bits - 1)) - 1)))
    return -mag if c & (1 << (bits - 1)) else mag


@pytest.mark.parametrize("fmt", [7, 8])
def test_bruteforce_tiny_groups_of_8(oracle, fmt):
    rng = np.random.default_rng(300 + fmt)
    c = oracle.fmt_constants(fmt)
    bits, m_fp, m_i = c["bits"], c["fp_max"], c["int_max"]
    k_exact = Fraction(m_fp).limit_denominator(1000) / m_i
    int_codes = [q & ((1 << bits) - 1) for q in range(-m_i, m_i + 1)]
    for trial in range(30):
        delta = 2.0 ** int(rng.integers(-3, 4))
        live = rng.uniform(-m_fp, m_fp, 3).astype(np.float32)
        live[int(rng.integers(0, 3))] = m_fp
        v = np.zeros(8, dtype=np.float32)
        v[:3] = live * np.float32(delta)
        codes, sb, e_fp, e_int = oracle.quantize_group(v, 1.0, fmt, oracle.SCALE_IN)
        assert len(codes) == 8 and oracle.e4m3_value(sb & 0x7F) == delta
        xs = [Fraction(float(t)) for t in live]
        best_fp = min(sum((_value(oracle, fmt, q, False) - x) ** 2 for q, x in zip(qs, xs))
                      for qs in itertools.product(range(1 << bits), repeat=3))
        best_int = min(sum((_value(oracle, fmt, q, True) * k_exact - x) ** 2 for q, x in zip(qs, xs))
                       for qs in itertools.product(int_codes, repeat=3))
        is_int = bool(sb & 0x80)
        chosen = sum((_value(oracle, fmt, q, is_int) * (k_exact if is_int else 1) - x) ** 2
                     for q, x in zip(codes[:3], xs))
        tol = Fraction(1, 10 ** 5) * max(best_fp, best_int, Fraction(1, 10 ** 30))
        assert all(q == 0 for q in codes[3:])
        assert chosen <= min(best_fp, best_int) + tol
        if abs(best_int - best_fp) > tol:
            assert is_int == (best_int < best_fp)


def _mse(oracle, fmt, xb, x):
    c, s, a = oracle.quantize(xb, fmt)
    return float(np.mean((oracle.dequantize(c, s, a, fmt, np.float64) - x) ** 2))


@pytest.mark.parametrize("fmt8,fmt16", PAIRS)
def test_smaller_blocks_lose_less(oracle, fmt8, fmt16):
    rng = np.random.default_rng(400)
    xb = oracle.bf16_bits(rng.standard_normal((64, 1024)))
    x = oracle.bf16_to_f32(xb).astype(np.float64)
    assert _mse(oracle, fmt8, xb, x) < 0.95 * _mse(oracle, fmt16, xb, x)


def test_if4_bs8_never_worse_than_nvfp4_bs8(oracle):
    rng = np.random.default_rng(401)
    xb = oracle.bf16_bits(rng.standard_t(3, (32, 512)))
    x = oracle.bf16_to_f32(xb).astype(np.float64)
    ci, si, ai = oracle.quantize(xb, 7)
    cn, sn, an = oracle.quantize(xb, 9)
    ei = ((oracle.dequantize(ci, si, ai, 7, np.float64) - x) ** 2).reshape(-1, 8).sum(1)
    en = ((oracle.dequantize(cn, sn, an, 9, np.float64) - x) ** 2).reshape(-1, 8).sum(1)
    assert np.all(ei <= en * (1 + 1e-5) + 1e-30) and np.mean(ei < en) > 0.1
    fp = (si.reshape(-1) & 0x80) == 0
    np.testing.assert_array_equal(si.reshape(-1)[fp], sn.reshape(-1)[fp])


def test_sr_uses_the_groups_own_counter(oracle):
    """Group gi of 8 rounds with the first 8 draws of Philox counter gi."""
    rng = np.random.default_rng(402)
    xb = oracle.bf16_bits(rng.standard_normal((4, 64)))
    c, s, a = oracle.quantize(xb, 7, oracle.SR, seed=77)
    v = oracle.bf16_to_f32(xb)
    for gi in (0, 5, 17, 31):
        r, g = divmod(gi, 8)
        codes, sb, _, _ = oracle.quantize_group(v[r, 8 * g:8 * g + 8], a, 7, oracle.SR,
                                                oracle.sr_bits(77, gi)[:8])
        assert sb == s[r, g]
        np.testing.assert_array_equal(oracle.unpack_group(7, c[r, 4 * g:4 * g + 4]), codes)
