"""Pins of the oracle's quantizer to the paper.

- Fig. 3a worked example (tests/golden/fig3a_worked_example.json), exact.
- Brute force over every code vector of tiny groups: the FP and INT
  candidates are the least-squares code vectors and the selection takes the
  type with the smaller error (Fig. 3a (selection)), checked in exact rationals.
- IF4's error never exceeds NVFP4's on the same group, and an IF4 group that
  keeps FP is bit-identical to the NVFP4 encoding (Sec. 3).
- Exact round trips of values already on the FP or scaled-INT grid (Eq. 1-2).
- Eq. 1: alpha = max|X| / (6 * 448); zero tensors; the strided (token) axis
  is the row-wise quantizer applied to the transpose.
"""
import itertools
import json
import os
from fractions import Fraction

import numpy as np
import pytest

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _group(values):
    v = np.zeros(16, dtype=np.float32)
    v[: len(values)] = values
    return v


def test_fig3a_worked_example_alpha_one(oracle):
    ex = _golden("fig3a_worked_example.json")
    v = _group(ex["X"])
    codes, sb, e_fp, e_int = oracle.quantize_group(v, 1.0, oracle.FMT_IF4, oracle.SCALE_IN)
    delta = oracle.e4m3_value(sb & 0x7F)
    assert delta == ex["line2_delta_e4m3"] == ex["line1_delta_before_cast"]
    # INT selected: sign bit of the scale set (Sec. 3), codes of the INT candidate
    assert sb & 0x80
    assert [int(c) for c in codes[:4]] == ex["line10_selected"] == ex["line7_int4_values"]
    assert all(c == 0 for c in codes[4:])
    # errors are kept in x-bar units; times Delta^2 they are the errors of Fig. 3a.
    # The printed 46.0 is the sum of squares (1 + 9 + 36 + 0), not the mean.
    assert e_fp * delta ** 2 == pytest.approx(ex["line6_fp_error_printed"], rel=1e-6)
    assert e_int * delta ** 2 == pytest.approx(ex["line9_int_error_printed"], abs=1e-9)
    # the FP candidate itself (NVFP4 stops at the FP candidate)
    nv_codes, nv_sb, _, _ = oracle.quantize_group(v, 1.0, oracle.FMT_NVFP4, oracle.SCALE_IN)
    fp_vals = [oracle.fp_magnitude(oracle.FMT_NVFP4, c & 7) for c in nv_codes[:4]]
    assert fp_vals == ex["line4_fp4_values"]
    assert nv_sb == sb & 0x7F
    # dequantized values of both candidates
    packed = oracle.pack_group(oracle.FMT_IF4, codes)[None, :]
    deq = oracle.dequantize(packed, np.array([[sb]], np.uint8), 1.0)[0, :4]
    assert list(deq) == ex["line8_int_dequant"]
    nv_packed = oracle.pack_group(oracle.FMT_NVFP4, nv_codes)[None, :]
    deq = oracle.dequantize(nv_packed, np.array([[nv_sb]], np.uint8), 1.0, oracle.FMT_NVFP4)[0, :4]
    assert list(deq) == ex["line5_fp_dequant"]


def test_fig3a_worked_example_auto_alpha(oracle):
    ex = _golden("fig3a_worked_example.json")
    x = oracle.bf16_bits(_group(ex["X"])[None, :])
    codes, scales, alpha = oracle.quantize(x)
    # Eq. 1: 42 / (6 * 448) = 2^-6 exactly; Eq. 2 then gives Delta = 448
    assert alpha == 42 / 2688 == 2.0 ** -6
    assert scales[0, 0] == 0x80 | 0x7E
    unpacked = oracle.unpack_group(oracle.FMT_IF4, codes[0])
    assert [int(c) for c in unpacked[:4]] == ex["line7_int4_values"]
    np.testing.assert_array_equal(oracle.dequantize(codes, scales, alpha)[0, :4],
                                  np.array(ex["X"], np.float32))


def _exact(x):
    return Fraction(float(x))


def _value_of_code(oracle, fmt, code, is_int):
    bits = oracle.BITS[fmt]
    if is_int:
        c = int(code)
        if c & (1 << (bits - 1)):
            c -= 1 << bits
        return c
    mag = Fraction(oracle.fp_magnitude(fmt, int(code) & ((1 << (bits - 1)) - 1)))
    return -mag if code & (1 << (bits - 1)) else mag


@pytest.mark.parametrize("fmt", [0, 2])
def test_bruteforce_tiny_groups(oracle, fmt):
    """Three live values, 13 zeros, Delta a power of two so x-bar = v / Delta
    exactly.  Every FP code vector (2^b)^3 and INT vector (2^b - 1)^3 is
    scored in exact rationals."""
    rng = np.random.default_rng(100 + fmt)
    c = oracle.fmt_constants(fmt)
    bits, m_fp, m_i = c["bits"], c["fp_max"], c["int_max"]
    k_exact = Fraction(m_fp).limit_denominator(1000) / m_i
    fp_codes = range(1 << bits)
    int_codes = [q & ((1 << bits) - 1) for q in range(-m_i, m_i + 1)]
    checked = 0
    for trial in range(40):
        j = int(rng.integers(-3, 4))
        delta = 2.0 ** j
        live = rng.uniform(-m_fp, m_fp, 3).astype(np.float32)
        live[int(rng.integers(0, 3))] = m_fp * np.sign(live[0] or 1.0)  # group max = M_FP
        if trial % 4 == 0:  # lattice values hit ties of both grids
            live = (np.round(live * 4) / 4).astype(np.float32)
            live[0] = m_fp
        v = _group(live * np.float32(delta))
        codes, sb, e_fp, e_int = oracle.quantize_group(v, 1.0, fmt, oracle.SCALE_IN)
        assert oracle.e4m3_value(sb & 0x7F) == delta
        xb = [Fraction(float(t)) for t in live]
        # exact least-squares over all code vectors
        best_fp = min(sum((_value_of_code(oracle, fmt, q, False) - x) ** 2 for q, x in zip(qs, xb))
                      for qs in itertools.product(fp_codes, repeat=3))
        best_int = min(sum((_value_of_code(oracle, fmt, q, True) * k_exact - x) ** 2
                           for q, x in zip(qs, xb))
                       for qs in itertools.product(int_codes, repeat=3))
        # the chosen candidate's exact error
        is_int = bool(sb & 0x80)
        chosen = sum((_value_of_code(oracle, fmt, q, is_int) * (k_exact if is_int else 1) - x) ** 2
                     for q, x in zip(codes[:3], xb))
        assert all(q == 0 for q in codes[3:])
        tol = Fraction(1, 10 ** 5) * max(best_fp, best_int, Fraction(1, 10 ** 30))
        assert chosen <= min(best_fp, best_int) + tol
        # selection: strict "<" in favour of INT (Fig. 3a (selection))
        if abs(best_int - best_fp) > tol:
            assert is_int == (best_int < best_fp)
        # the fp32 errors track the exact ones
        assert abs(Fraction(float(e_fp)) - best_fp) <= tol + Fraction(1, 10 ** 5) * best_fp
        checked += 1
    assert checked == 40


def test_if4_never_worse_than_nvfp4(oracle):
    rng = np.random.default_rng(3)
    x = rng.standard_t(3, size=(64, 256)).astype(np.float32)
    x[:, ::37] *= 20
    xb = oracle.bf16_bits(x)
    xf = oracle.bf16_to_f32(xb).astype(np.float64)
    c_if, s_if, a_if = oracle.quantize(xb, oracle.FMT_IF4)
    c_nv, s_nv, a_nv = oracle.quantize(xb, oracle.FMT_NVFP4)
    assert a_if == a_nv
    d_if = oracle.dequantize(c_if, s_if, a_if, oracle.FMT_IF4, np.float64)
    d_nv = oracle.dequantize(c_nv, s_nv, a_nv, oracle.FMT_NVFP4, np.float64)
    e_if = ((d_if - xf) ** 2).reshape(-1, 16).sum(1)
    e_nv = ((d_nv - xf) ** 2).reshape(-1, 16).sum(1)
    assert np.all(e_if <= e_nv * (1 + 1e-5) + 1e-30)
    assert np.mean(e_if < e_nv) > 0.2
    # FP groups of IF4 are bit-identical to the NVFP4 encoding
    fp_groups = (s_if.reshape(-1) & 0x80) == 0
    np.testing.assert_array_equal(s_if.reshape(-1)[fp_groups], s_nv.reshape(-1)[fp_groups])
    np.testing.assert_array_equal(c_if.reshape(-1, 8)[fp_groups], c_nv.reshape(-1, 8)[fp_groups])
    assert fp_groups.any() and (~fp_groups).any()


def test_roundtrip_fp_grid(oracle):
    """x = alpha * Delta * q with alpha = 2^k, Delta in E4M3 and q on the FP4
    grid (group max 6) is reproduced exactly."""
    rng = np.random.default_rng(11)
    grid = oracle.fp_grid(oracle.FMT_IF4)
    k = -3
    alpha = 2.0 ** k
    rows = []
    deltas = [448.0] + [oracle.e4m3_value(c) for c in rng.integers(1, 127, 31)]
    for d in deltas:
        q = rng.choice(grid, 16) * rng.choice([-1, 1], 16)
        q[rng.integers(0, 16)] = 6.0
        q[rng.integers(0, 16)] = 1.5   # no scaled-INT value fits 1.5: keeps the group FP
        rows.append(alpha * d * q)
    x = np.array(rows).reshape(4, 128)
    xb = oracle.bf16_bits(x)
    assert np.array_equal(oracle.bf16_to_f32(xb), x.astype(np.float32))
    codes, scales, a = oracle.quantize(xb)
    assert a == alpha
    assert np.all((scales & 0x80) == 0)
    np.testing.assert_array_equal(oracle.dequantize(codes, scales, a), x.astype(np.float32))


def test_roundtrip_int_grid(oracle):
    """Delta = 7 * 2^j and x = alpha * 6 * 2^j * q_int with max |q_int| = 7:
    the INT candidate is exact and selected (generalises Fig. 3a)."""
    rng = np.random.default_rng(12)
    rows = []
    for g in range(32):
        j = int(rng.integers(-4, 5))
        q = rng.integers(-7, 8, 16)
        q[rng.integers(0, 16)] = 7
        q[rng.integers(0, 16)] = 5   # 6*5/7 is not on the FP4 grid: keeps the group INT
        rows.append(6.0 * 2.0 ** j * q)
    x = np.array(rows, dtype=np.float64).reshape(8, 64)
    xb = oracle.bf16_bits(x)
    assert np.array_equal(oracle.bf16_to_f32(xb), x.astype(np.float32))
    codes, scales, a = oracle.quantize(xb, flags=oracle.SCALE_IN, tensor_scale=1.0)
    assert np.all(scales & 0x80)
    np.testing.assert_array_equal(oracle.dequantize(codes, scales, a), x.astype(np.float32))


def test_tensor_scale_eq1(oracle):
    assert oracle.tensor_scale(oracle.FMT_IF4, 2688.0) == 1.0
    assert oracle.tensor_scale(oracle.FMT_IF3, 4 * 448.0) == 1.0
    assert oracle.tensor_scale(oracle.FMT_IF6_E3M2, 28 * 448.0) == 1.0
    # gradient margin (Sec. 4.1): M_FP * 16/17 in place of M_FP
    a = oracle.tensor_scale(oracle.FMT_IF4, 1.0, oracle.MARGIN)
    assert a == np.float32(1.0) / (np.float32(6 * 16 / 17) * np.float32(448))


@pytest.mark.parametrize("fmt", [0, 1, 2, 3, 4])
def test_zero_tensor(oracle, fmt):
    xb = np.zeros((3, 32), np.uint16)
    codes, scales, a = oracle.quantize(xb, fmt)
    assert a == 0.0 and not codes.any() and not scales.any()
    assert not oracle.dequantize(codes, scales, a, fmt).any()


@pytest.mark.parametrize("flags", [0, 1, 2, 3, 7])
def test_strided_axis_is_transpose(oracle, flags):
    rng = np.random.default_rng(5)
    x = oracle.bf16_bits(rng.laplace(0, 1e-3, (64, 48)))
    c1, s1, a1 = oracle.quantize(x, flags=flags | oracle.STRIDED, rht_signs=0xA5C3, seed=9)
    c2, s2, a2 = oracle.quantize(np.ascontiguousarray(x.T), flags=flags, rht_signs=0xA5C3, seed=9)
    assert a1 == a2
    np.testing.assert_array_equal(s1, s2)
    np.testing.assert_array_equal(c1, c2)


def test_table1_max_min_values(oracle):
    t = _golden("table1_formats.json")["rows"]
    fp_max = oracle.fp_grid(oracle.FMT_IF4)[-1]
    fp_min = oracle.fp_grid(oracle.FMT_IF4)[1]
    e_max = oracle.e4m3_value(0x7E)
    e_min = oracle.e4m3_value(0x01)
    for name in ("NVFP4", "IF4"):
        assert fp_max * e_max == t[name]["max"][0] * t[name]["max"][1]
        assert fp_min * e_min == t[name]["min"][0] * 2.0 ** t[name]["min"][1]
    assert 7 * e_max == t["NVINT4"]["max"][0] * t["NVINT4"]["max"][1]


def test_selection_tie_goes_to_fp(oracle):
    """Fig. 3a (selection) takes INT only when its error is strictly smaller.
    An outlier group whose small values round to zero in both candidates
    gives bit-identical fp32 errors (the max is exact in both, and the INT
    max's 7*fp32(6/7) - 6 residue is absorbed by the larger sum), so the
    group must stay FP."""
    v = _group([6.0, 0.1, -0.2, 0.05, 0.15, -0.12, 0.07, 0.2])
    codes, sb, e_fp, e_int = oracle.quantize_group(v, 1.0, oracle.FMT_IF4, oracle.SCALE_IN)
    assert e_fp == e_int and e_fp > 0
    assert sb == oracle.e4m3_encode(1.0)          # FP: sign bit clear
    assert codes[0] == 7 and all(c in (0, 8) for c in codes[1:])
