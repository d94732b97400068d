"""Pins of the oracle's random Hadamard transform, stochastic rounding and
counter-based generator.

- RHT (Sec. 1, Sec. 4.1): the butterfly equals (1/4) H16 diag(s) with H16
  built from its plain definition H[i][j] = (-1)^popcount(i & j); it is
  orthonormal, exact on small integers, and a pair of transformed GEMM
  operands gives the untransformed product.
- SR (Sec. 1, App. B): NVFP4 with SR is unbiased inside the range; IF4 with
  SR moves large values up in magnitude, the bias App. B describes.
- Philox4x32-10: the oracle's stream equals rocRAND's independent
  implementation (a library routine, compiled here from its header).
"""
import os
import shutil
import subprocess

import numpy as np
import pytest


def _hadamard16():
    i = np.arange(16)
    pc = np.vectorize(lambda t: bin(t).count("1"))(i[:, None] & i[None, :])
    return np.where(pc % 2 == 0, 1.0, -1.0)


def test_rht_matrix_is_scaled_sylvester_hadamard(oracle):
    H = _hadamard16()
    M = np.stack([oracle.rht16(np.eye(16, dtype=np.float32)[j], 0) for j in range(16)], 1)
    np.testing.assert_array_equal(M, 0.25 * H)
    np.testing.assert_array_equal(M @ M.T, np.eye(16))


def test_rht_signs_and_random_inputs(oracle):
    H = _hadamard16()
    rng = np.random.default_rng(1)
    for trial in range(200):
        signs = int(rng.integers(0, 1 << 16))
        s = np.array([-1.0 if (signs >> j) & 1 else 1.0 for j in range(16)])
        if trial < 50:
            x = rng.integers(-100, 100, 16).astype(np.float32)   # exact in fp32
        else:
            x = (rng.standard_normal(16) * 10.0 ** rng.uniform(-3, 3)).astype(np.float32)
        ref = 0.25 * H @ (s * x.astype(np.float64))
        got = oracle.rht16(x, signs).astype(np.float64)
        if trial < 50:
            np.testing.assert_array_equal(got, ref)
        else:
            # 4 rounded additions on values bounded by sum|x|
            assert np.max(np.abs(got - ref)) <= 4 * 2.0 ** -24 * np.abs(x).sum()


def test_rht_paired_gemm_invariance(oracle):
    rng = np.random.default_rng(2)
    A = rng.standard_normal((8, 64)).astype(np.float32)
    B = rng.standard_normal((5, 64)).astype(np.float32)
    signs = 0xB38D
    TA = np.stack([np.concatenate([oracle.rht16(r[g:g + 16], signs) for g in range(0, 64, 16)])
                   for r in A])
    TB = np.stack([np.concatenate([oracle.rht16(r[g:g + 16], signs) for g in range(0, 64, 16)])
                   for r in B])
    np.testing.assert_allclose(TA.astype(np.float64) @ TB.T.astype(np.float64),
                               A.astype(np.float64) @ B.T.astype(np.float64), atol=1e-4)


def _sr_trials(oracle, fmt, v, trials, seed0=0, flags=0):
    """Dequantized values of one group over `trials` Philox seeds (alpha=1)."""
    out = np.zeros((trials, 16))
    for t in range(trials):
        h = oracle.sr_bits(seed0 + t, 0)
        codes, sb, _, _ = oracle.quantize_group(v, 1.0, fmt, oracle.SCALE_IN | oracle.SR | flags, h)
        packed = oracle.pack_group(fmt, codes)[None, :]
        out[t] = oracle.dequantize(packed, np.array([[sb]], np.uint8), 1.0, fmt, np.float64)[0]
    return out


def test_sr_nvfp4_unbiased(oracle):
    v = np.array([6.0, 0.3, 1.2, -2.7, 4.9, -3.3, 0.05, 5.5, -0.8, 2.2, 3.9, -1.6,
                  0.7, -4.2, 1.9, 0.0], np.float32)
    trials = 4000
    deq = _sr_trials(oracle, oracle.FMT_NVFP4, v, trials)
    mean = deq.mean(0)
    # per-element spread is at most half the local grid step (2 near 6)
    sem = np.maximum(deq.std(0), 1e-3) / np.sqrt(trials)
    assert np.all(np.abs(mean - v) <= 5 * sem + 1e-4), (mean - v) / sem
    # grid points and the maximum are kept exactly
    assert np.all(deq[:, 0] == 6.0) and np.all(deq[:, 15] == 0.0)


def _group_max_bias(oracle, fmt, flags, groups=80, trials=150):
    """Mean signed change of each group's largest value, in units of it, over
    Laplace groups whose E4M3 scale is not exact (Delta_raw in [1, 2))."""
    rng = np.random.default_rng(5)
    bias = []
    for g in range(groups):
        v = rng.laplace(0, 1, 16)
        v = (v * 6 * rng.uniform(1, 2) / np.abs(v).max()).astype(np.float32)
        i = int(np.argmax(np.abs(v)))
        d = _sr_trials(oracle, fmt, v, trials, seed0=1000 * g, flags=flags)
        bias.append((d[:, i].mean() - v[i]) * np.sign(v[i]) / abs(v[i]))
    return np.mean(bias), np.std(bias) / np.sqrt(groups)


def test_sr_margin_removes_scale_saturation_bias(oracle):
    """Sec. 4.1: without the 16/17 factor a group maximum whose E4M3 scale
    rounded down saturates, biasing NVFP4-SR down; with it NVFP4-SR is
    unbiased."""
    m0, s0 = _group_max_bias(oracle, oracle.FMT_NVFP4, 0)
    m1, s1 = _group_max_bias(oracle, oracle.FMT_NVFP4, oracle.MARGIN)
    assert m0 < -4 * s0
    assert abs(m1) < 3 * s1 + 1e-3


def test_sr_if4_biases_large_values_up(oracle):
    """App. B: selecting between the two SR candidates by error moves the
    largest values up in magnitude (a few percent of the group maximum),
    where NVFP4-SR with the same margin stays unbiased."""
    m_if, s_if = _group_max_bias(oracle, oracle.FMT_IF4, oracle.MARGIN)
    m_nv, s_nv = _group_max_bias(oracle, oracle.FMT_NVFP4, oracle.MARGIN)
    assert m_if > 6 * s_if and 0.005 < m_if < 0.08
    assert m_if - m_nv > 4 * np.hypot(s_if, s_nv)


def test_sr_rtn_type_is_unbiased(oracle):
    """App. B's alternative: decide FP or INT on the round-to-nearest
    candidates, then round stochastically in that type.  The type no longer
    depends on the random draws (every trial keeps the RTN scale byte), the
    group is unbiased element by element, and the upward bias of the largest
    values that the default IF4-SR shows disappears."""
    v = np.array([6.0, 0.3, 1.2, -2.7, 4.9, -3.3, 0.05, 5.5, -0.8, 2.2, 3.9, -1.6,
                  0.7, -4.2, 1.9, 0.0], np.float32)
    _, sb_rtn, _, _ = oracle.quantize_group(v, 1.0, oracle.FMT_IF4, oracle.SCALE_IN)
    for t in range(50):
        h = oracle.sr_bits(t, 0)
        _, sb, _, _ = oracle.quantize_group(v, 1.0, oracle.FMT_IF4,
                                            oracle.SCALE_IN | oracle.SR | oracle.SR_RTN_TYPE, h)
        assert sb == sb_rtn
    trials = 4000
    deq = _sr_trials(oracle, oracle.FMT_IF4, v, trials, flags=oracle.SR_RTN_TYPE)
    sem = np.maximum(deq.std(0), 1e-3) / np.sqrt(trials)
    assert np.all(np.abs(deq.mean(0) - v) <= 5 * sem + 1e-4), (deq.mean(0) - v) / sem
    m, s = _group_max_bias(oracle, oracle.FMT_IF4, oracle.MARGIN | oracle.SR_RTN_TYPE)
    assert abs(m) < 3 * s + 1e-3, (m, s)


def test_sr_rtn_type_without_sr_is_plain_rtn(oracle):
    rng = np.random.default_rng(17)
    for _ in range(200):
        v = (rng.standard_t(3, 16) * rng.uniform(0.1, 10)).astype(np.float32)
        a = oracle.quantize_group(v, 1.0, oracle.FMT_IF4, oracle.SCALE_IN)
        b = oracle.quantize_group(v, 1.0, oracle.FMT_IF4, oracle.SCALE_IN | oracle.SR_RTN_TYPE)
        assert np.array_equal(a[0], b[0]) and a[1] == b[1]


def test_sr_bits_layout(oracle):
    seed, group = 0x0123456789ABCDEF, 77
    key = [seed & 0xFFFFFFFF, seed >> 32]
    w = np.concatenate([oracle.philox4x32_10([group, 0, b, 0], key) for b in (0, 1)])
    h = oracle.sr_bits(seed, group)
    for j in range(16):
        assert h[j] == (int(w[j >> 1]) >> (16 * (j & 1))) & 0xFFFF


ROCRAND_PROBE = r"""
#include <hip/hip_runtime.h>
#include <rocrand/rocrand_philox4x32_10.h>
#include <cstdio>
#include <cstdlib>
int main(int argc, char** argv) {
  // argv: seed subsequence offset_blocks
  unsigned long long seed = strtoull(argv[1], 0, 0), sub = strtoull(argv[2], 0, 0),
                     off = strtoull(argv[3], 0, 0);
  rocrand_device::philox4x32_10_engine e(seed, sub, 4 * off);
  uint4 v = e.next4();
  printf("%u %u %u %u\n", v.x, v.y, v.z, v.w);
  return 0;
}
"""


@pytest.fixture(scope="module")
def rocrand_probe(tmp_path_factory):
    hipcc = shutil.which("hipcc") or "/opt/rocm/bin/hipcc"
    if not os.path.exists(hipcc):
        pytest.skip("hipcc not available")
    d = tmp_path_factory.mktemp("rocrand")
    src = d / "probe.cpp"
    src.write_text(ROCRAND_PROBE)
    exe = d / "probe"
    subprocess.run([hipcc, "-x", "hip", "--offload-arch=gfx950", "-O1", str(src), "-o", str(exe)],
                   check=True, capture_output=True)
    return str(exe)


def test_philox_matches_rocrand(oracle, rocrand_probe):
    """rocRAND's engine(seed, subsequence, 4*n) emits Philox4x32-10 of the
    counter (n_lo, n_hi, sub_lo, sub_hi) under key (seed_lo, seed_hi)."""
    rng = np.random.default_rng(8)
    cases = [(0, 0, 0), (0xFFFFFFFFFFFFFFFF, 1, 3), (0x0123456789ABCDEF, 1, 5)]
    cases += [(int(rng.integers(0, 2 ** 63)), int(rng.integers(0, 2)), int(rng.integers(0, 2 ** 40)))
              for _ in range(12)]
    for seed, sub, n in cases:
        out = subprocess.run([rocrand_probe, str(seed), str(sub), str(n)], check=True,
                             capture_output=True, text=True).stdout.split()
        ref = [int(t) for t in out]
        got = oracle.philox4x32_10([n & 0xFFFFFFFF, n >> 32, sub & 0xFFFFFFFF, sub >> 32],
                                   [seed & 0xFFFFFFFF, seed >> 32])
        assert [int(t) for t in got] == ref, (seed, sub, n)
