"""Arithmetic identities the quantizer kernels use in place of the
straightforward forms, checked on the CPU in binary32
(tests/arith/kernel_identities.c, built here with gcc -ffp-contract=off):

- stochastic rounding as ceil(t - u) of the exact ratio, against
  "floor + 1 iff u * step < m - floor" on the E2M1, E2M3, E3M2 and E2M0
  grids and the INT candidates, every sampled fp32 magnitude of each range
  with the draws at, below and above its fraction;
- the group-scale quotient by Markstein's correction, against the correctly
  rounded division, as the E4M3 encoder consumes it;
- the GEMM's INT6 decode (IF6): each pair of six-bit two's-complement codes
  taken from one 16-bit half of a word or of an aligned copy, shifted per
  lane, masked, its sign bit flipped under the exponent of 1024 and 1056
  subtracted, against the codes read by their definition (code j at bits
  6j .. 6j + 5 of the group's 96 bits), for every 12-bit pair value;
- the GEMM's IF3 selector spread: four 3-bit codes to one byte each by a
  packed 16-bit shift, a word shift and two masks, against the codes read
  by their definition, for every 16-bit input under random upper bits.

The sampled strides keep this to a few seconds; stride 1 (every value) was
run too and found no difference."""
import os
import shutil
import subprocess

import numpy as np
import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "arith", "kernel_identities.c")


@pytest.fixture(scope="module")
def checker(tmp_path_factory):
    if shutil.which("gcc") is None:
        pytest.skip("gcc not available")
    exe = str(tmp_path_factory.mktemp("arith") / "kernel_identities")
    subprocess.run(["gcc", "-O2", "-ffp-contract=off", "-o", exe, SRC, "-lm"], check=True)
    return exe


@pytest.mark.parametrize("what, stride", [("sr", 97), ("div", 61)])
def test_kernel_identity(checker, what, stride):
    out = subprocess.run([checker, what, str(stride)], capture_output=True, text=True)
    assert out.returncode == 0, out.stdout + out.stderr
    n, bad = (int(w) for w in out.stdout.split()[1::2][:2])
    assert bad == 0 and n > 10 ** 8, out.stdout


# (source, half, S0, S1) of pair i in the IF6 GEMM decode: the source is a
# word of the group (w0, w1, w2) or one of the aligned copies xa = bits 8-39
# and xb = bits 56-87 of the 96-bit group
INT6_PAIRS = [("w0", 0, 0, 6), ("xa", 0, 4, 10), ("xa", 1, 0, 6), ("w1", 0, 4, 10),
              ("w1", 1, 0, 6), ("xb", 0, 4, 10), ("xb", 1, 0, 6), ("w2", 1, 4, 10)]


def _int6_pair_kernel(x, hi, s0, s1):
    """Lanes (code 2i, code 2i + 1) as the kernel forms them, in float16."""
    s = ((x >> np.uint64(16)) if hi else x) & np.uint64(0xFFFF)
    lo = ((s >> np.uint64(s0)) & np.uint64(0x3F)) ^ np.uint64(0x6420)
    up = ((s >> np.uint64(s1)) & np.uint64(0x3F)) ^ np.uint64(0x6420)
    f = lambda b: b.astype(np.uint16).view(np.float16)
    return f(lo) - np.float16(1056.0), f(up) - np.float16(1056.0)


def test_int6_pair_decode():
    rng = np.random.default_rng(7)
    n = 4096 * 8
    # every 12-bit value at every pair position, the other bits random
    bits = [rng.integers(0, 2 ** 32, n, dtype=np.uint64) for _ in range(3)]
    pair = np.tile(np.arange(4096, dtype=np.uint64), 8)
    pos = np.repeat(np.arange(8), 4096)
    stream = [(b0 | (b1 << np.uint64(32)), b2) for b0, b1, b2 in [bits]][0]
    lo64, hi32 = stream
    for i in range(8):
        sel = pos == i
        sh = 12 * i
        if sh + 12 <= 64:
            m = np.uint64(0xFFF) << np.uint64(sh)
            lo64[sel] = (lo64[sel] & ~m) | (pair[sel] << np.uint64(sh))
        elif sh >= 64:
            m = np.uint64(0xFFF) << np.uint64(sh - 64)
            hi32[sel] = (hi32[sel] & ~m) | (pair[sel] << np.uint64(sh - 64))
        else:  # pair 5 spans bits 60-71
            k = 64 - sh
            lo64[sel] = (lo64[sel] & ~(np.uint64((1 << k) - 1) << np.uint64(sh))) | \
                ((pair[sel] & np.uint64((1 << k) - 1)) << np.uint64(sh))
            hi32[sel] = (hi32[sel] & ~np.uint64((1 << (12 - k)) - 1)) | (pair[sel] >> np.uint64(k))
    m32 = np.uint64(0xFFFFFFFF)
    w0, w1, w2 = lo64 & m32, lo64 >> np.uint64(32), hi32 & m32
    src = {"w0": w0, "w1": w1, "w2": w2,
           "xa": (lo64 >> np.uint64(8)) & m32,
           "xb": ((lo64 >> np.uint64(56)) | (w2 << np.uint64(8))) & m32}

    def code(j):  # the definition: six bits at 6j of the 96-bit group, two's complement
        b = 6 * j
        v = (lo64 >> np.uint64(b)) if b + 6 <= 64 else \
            ((lo64 >> np.uint64(b)) | (hi32 << np.uint64(64 - b))) if b < 64 else (hi32 >> np.uint64(b - 64))
        v = (v & np.uint64(0x3F)).astype(np.int64)
        return np.where(v >= 32, v - 64, v)

    checked = 0
    for i, (name, hi, s0, s1) in enumerate(INT6_PAIRS):
        a, b = _int6_pair_kernel(src[name], hi, s0, s1)
        assert np.array_equal(a.astype(np.int64), code(2 * i)), i
        assert np.array_equal(b.astype(np.int64), code(2 * i + 1)), i
        assert not np.signbit(a[code(2 * i) == 0]).any()
        checked += int((pos == i).sum())
    assert checked == n


def test_if3_selector_spread():
    rng = np.random.default_rng(11)
    t = np.arange(1 << 16, dtype=np.uint64) | (rng.integers(0, 1 << 16, 1 << 16, dtype=np.uint64) << np.uint64(16))
    s = t & np.uint64(0xFFFF)
    y = s | ((s >> np.uint64(6)) << np.uint64(16))           # lanes: s >> 0, s >> 6
    got = (y & np.uint64(0x00070007)) | (((y << np.uint64(5)) & np.uint64(0xFFFFFFFF)) & np.uint64(0x07000700))
    want = sum(((t >> np.uint64(3 * k)) & np.uint64(7)) << np.uint64(8 * k) for k in range(4))
    assert np.array_equal(got, want)
