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
