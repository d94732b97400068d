"""Pins of the oracle's element and scale codecs to what the paper fixes.

- FP4 E2M1 grid +-{0, 0.5, 1, 1.5, 2, 3, 4, 6} (Sec. 1).
- E4M3 scale: largest value 448 (Sec. 3), smallest 2^-9 (Table 1's minimum
  value 0.5 x 2^-9 is the smallest FP4 value times the smallest scale);
  every code cross-checked against torch.float8_e4m3fn (a library routine).
- IF3 / IF6 element types (Table 6) and the INT/FP range ratios 6/7, 4/3,
  7.5/31, 28/31 (Sec. 3 and the Sec. 5.1 footnote).
- Round-to-nearest ties resolve to the even code (the meaning of RNE).
- Packing: bits per parameter 3.5 / 4.5 / 6.5 (Table 6).
"""
from fractions import Fraction

import numpy as np
import pytest
import torch


def test_fp4_grid_matches_paper(oracle):
    assert list(oracle.fp_grid(oracle.FMT_IF4)) == [0, 0.5, 1, 1.5, 2, 3, 4, 6]
    assert list(oracle.fp_grid(oracle.FMT_NVFP4)) == [0, 0.5, 1, 1.5, 2, 3, 4, 6]


def test_other_element_types(oracle):
    # E2M0 (IF3's FP type): 0, 1, 2, 4
    assert list(oracle.fp_grid(oracle.FMT_IF3)) == [0, 1, 2, 4]
    # E2M3 spans 0..7.5 in steps of 1/8 below 2; E3M2 reaches 28
    g = oracle.fp_grid(oracle.FMT_IF6_E2M3)
    assert g[-1] == 7.5 and g[1] == 0.125 and len(g) == 32
    g = oracle.fp_grid(oracle.FMT_IF6_E3M2)
    assert g[-1] == 28 and g[1] == 0.0625 and len(g) == 32
    # all grids strictly increasing
    for fmt in range(5):
        g = oracle.fp_grid(fmt)
        assert np.all(np.diff(g) > 0)


@pytest.mark.parametrize("fmt,ratio,int_max", [
    (0, Fraction(6, 7), 7), (2, Fraction(4, 3), 3),
    (3, Fraction(15, 62), 31), (4, Fraction(28, 31), 31)])
def test_range_alignment_ratios(oracle, fmt, ratio, int_max):
    c = oracle.fmt_constants(fmt)
    assert c["int_max"] == int_max
    # k_dn is the fp32 nearest to M_FP/M_I (Sec. 5.1 footnote), c_up to its inverse
    for val, exact in ((c["k_dn"], ratio), (c["c_up"], 1 / ratio)):
        f = np.float32(val)
        ulp = Fraction(float(np.spacing(f)))
        assert abs(Fraction(float(f)) - exact) <= ulp / 2


def test_e4m3_all_codes_vs_torch(oracle):
    codes = torch.arange(127, dtype=torch.uint8)
    ref = codes.view(torch.float8_e4m3fn).float().tolist()
    got = [oracle.e4m3_value(c) for c in range(127)]
    assert got == ref
    assert max(got) == 448.0                       # Sec. 3: M_FP8 = 448
    assert min(v for v in got if v > 0) == 2.0 ** -9  # Table 1 minimum / 0.5


def test_e4m3_encode_vs_torch(oracle):
    rng = np.random.default_rng(7)
    xs = np.concatenate([
        np.exp2(rng.uniform(-13, 9, 4000)),
        np.array([oracle.e4m3_value(c) for c in range(127)]),
        # midpoints between neighbouring codes (ties)
        np.array([(oracle.e4m3_value(c) + oracle.e4m3_value(c + 1)) / 2 for c in range(126)]),
        [0.0, 2.0 ** -10, 2.0 ** -10 * 1.0001, 448.0, 463.9, 464.0]]).astype(np.float32)
    xs = xs[xs <= 464.0]
    ref = torch.from_numpy(xs).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    got = np.array([oracle.e4m3_encode(float(x)) for x in xs])
    np.testing.assert_array_equal(got, ref)


def test_e4m3_saturates(oracle):
    # above 464 torch produces NaN; a scale must stay finite, so it saturates to 448
    for x in (465.0, 500.0, 1e6, 3.0e38):
        assert oracle.e4m3_encode(x) == 0x7E


@pytest.mark.parametrize("m,idx", [
    (0.25, 0), (0.75, 2), (1.25, 2), (1.75, 4), (2.5, 4), (3.5, 6), (5.0, 6),
    (0.2499, 0), (0.2501, 1), (5.01, 7), (6.0, 7), (7.0, 7), (1e30, 7)])
def test_fp4_round_to_nearest_even(oracle, m, idx):
    assert oracle.fp_round_index(oracle.FMT_IF4, m) == idx


def test_e2m0_ties(oracle):
    # IF3 grid 0,1,2,4: ties 0.5->0, 1.5->2, 3->2 (even code index)
    assert [oracle.fp_round_index(oracle.FMT_IF3, m) for m in (0.5, 1.5, 3.0, 9.0)] == [0, 2, 2, 3]


def test_pack_low_nibble_first(oracle):
    codes = np.arange(16, dtype=np.uint8)
    packed = oracle.pack_group(oracle.FMT_IF4, codes)
    assert list(packed) == [0x10, 0x32, 0x54, 0x76, 0x98, 0xBA, 0xDC, 0xFE]


@pytest.mark.parametrize("fmt,bits_per_param", [(2, 3.5), (0, 4.5), (3, 6.5), (4, 6.5)])
def test_pack_roundtrip_and_density(oracle, fmt, bits_per_param):
    rng = np.random.default_rng(fmt)
    bits = oracle.BITS[fmt]
    for _ in range(50):
        codes = rng.integers(0, 1 << bits, 16, dtype=np.uint8)
        packed = oracle.pack_group(fmt, codes)
        assert packed.size * 8 == 16 * bits
        np.testing.assert_array_equal(oracle.unpack_group(fmt, packed), codes)
    # Table 6: code bits plus one 8-bit scale per 16 values
    assert (16 * bits + 8) / 16 == bits_per_param


def _bf16_nearest_even_by_definition(f32: np.ndarray) -> np.ndarray:
    """bf16 bit patterns of finite fp32 values from the definition of
    round-to-nearest-even: of the two bf16 numbers that bracket x (its
    truncation toward zero and the next one away from zero), take the
    nearer, measured exactly in fp64, and on a tie the one with the even
    significand.  The largest finite bf16 rounds to infinity when the
    next step would be reached."""
    x = np.asarray(f32, dtype=np.float32)
    u = x.view(np.uint32).astype(np.int64)
    lo = (u >> 16) & 0xFFFF                       # truncation toward zero
    hi = lo + 1                                   # next bf16 away from zero (sign kept)

    def val(b):
        return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)

    xv = x.astype(np.float64)
    mag_hi = np.where((hi & 0x7FFF) >= 0x7F80, np.inf, 0.0)
    d_lo = np.abs(xv - val(lo))
    vh = np.where(np.isinf(mag_hi), np.copysign(2.0 ** 128, xv), val(np.where((hi & 0x7FFF) >= 0x7F80, lo, hi)))
    d_hi = np.abs(vh - xv)
    pick_hi = (d_hi < d_lo) | ((d_hi == d_lo) & ((lo & 1) == 1))
    return np.where(pick_hi, hi, lo).astype(np.uint16)


def test_bf16_rounding_against_definition_and_torch(oracle):
    """oracle.bf16_bits (the bf16 round-to-nearest-even behind every
    expected bf16 output) against torch's float -> bfloat16 conversion and
    against the rounding definition evaluated exactly: random finite fp32
    bit patterns over every exponent, exact ties with even and odd
    truncations, values one ulp either side of a tie, fp32 subnormals and
    values near the bf16 overflow threshold (which round to infinity)."""
    rng = np.random.default_rng(7)
    u = rng.integers(0, 1 << 32, 1 << 20, dtype=np.uint64).astype(np.uint32)
    u = u[(u & 0x7F800000) != 0x7F800000]                       # finite only
    base = rng.integers(0, 1 << 16, 1 << 16, dtype=np.uint64).astype(np.uint32) << 16
    base = base[(base & 0x7F800000) != 0x7F800000]
    ties = base | 0x8000
    near = np.concatenate([ties - 1, ties + 1])
    sub = rng.integers(0, 1 << 23, 1 << 14, dtype=np.uint64).astype(np.uint32)
    sub = np.concatenate([sub, sub | 0x80000000, np.array([0x00008000, 0x00018000, 0x80008000], np.uint32)])
    top = np.arange(0x7F7F0000, 0x7F800000, 7, dtype=np.uint32)
    top = np.concatenate([top, top | 0x80000000, np.array([0x7F7F7FFF, 0x7F7F8000, 0x7F7FFFFF], np.uint32)])
    x = np.concatenate([u, ties, near, sub, top]).view(np.float32)
    got = oracle.bf16_bits(x)
    want_torch = torch.from_numpy(x.copy()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(got, want_torch)
    np.testing.assert_array_equal(got, _bf16_nearest_even_by_definition(x))
    # spot values: a tie with an even truncation stays, an odd one rounds up
    assert oracle.bf16_bits(np.array([1.0 + 2.0 ** -8], np.float32))[0] == 0x3F80
    assert oracle.bf16_bits(np.array([1.0 + 3 * 2.0 ** -8], np.float32))[0] == 0x3F82
    assert oracle.bf16_bits(np.array([np.float32(3.4e38)], np.float32))[0] == 0x7F80
