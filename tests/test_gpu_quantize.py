"""GPU parity of the quantizer and the dequantizer: codes, scale bytes,
alpha and dequantized values bit-identical to the CPU oracle, for every
format and flag combination, ragged and degenerate shapes, adversarial ties,
and the distributions of the measured workloads."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2603_28765_amd import ops, workloads
from tests.gpu_common import (FORMATS, assert_quant_equal, bits, gpu_quantize, require_gpu)

pytestmark = pytest.mark.gpu

FLAG_SETS = [0, ops.RHT, ops.SR, ops.MARGIN_16_17, ops.RHT | ops.SR | ops.MARGIN_16_17,
             ops.SR | ops.SR_RTN_TYPE, ops.RHT | ops.SR | ops.MARGIN_16_17 | ops.SR_RTN_TYPE]


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def rand_bf16(shape, seed, kind="normal"):
    rng = np.random.default_rng(seed)
    if kind == "normal":
        x = rng.standard_normal(shape)
    elif kind == "outliers":
        x = rng.standard_t(3, shape) * 0.5
        x[..., :: max(1, shape[-1] // 5)] *= 50
    elif kind == "wide":
        x = rng.standard_normal(shape) * np.exp2(rng.uniform(-30, 30, shape))
    return workloads.to_bf16(x)


def test_tiny_config_if4_rtn():
    """The 256x256 N(0,1) case (seed 0), both operands, IF4 round-to-nearest."""
    w = workloads.tiny()
    for name in ("A", "B"):
        assert_quant_equal(ops.IF4, w.tensors[name], tag=f"tiny {name}")


@pytest.mark.parametrize("fmt", FORMATS)
@pytest.mark.parametrize("flags", FLAG_SETS)
def test_rowwise_all_formats_and_flags(fmt, flags):
    for shape, kind, seed in [((37, 48), "normal", 1), ((130, 4096), "outliers", 2),
                              ((1, 16), "normal", 3), ((64, 272), "wide", 4)]:
        x = rand_bf16(shape, seed + 10 * fmt, kind)
        assert_quant_equal(fmt, x, flags, signs=0xA5C3, seed=12345,
                           tag=f"fmt {fmt} flags {flags} {shape} {kind}")


@pytest.mark.parametrize("fmt", FORMATS)
@pytest.mark.parametrize("flags", FLAG_SETS)
def test_strided_axis(fmt, flags):
    # 4-bit formats with cols % 8 == 0 and rows % 256 == 0 take the register
    # path (here (512, 1032), with a partial last 64-column tile); the other
    # shapes and formats the LDS-tile path
    for shape, kind, seed in [((48, 37), "normal", 5), ((256, 100), "outliers", 6),
                              ((16, 1), "normal", 7), ((128, 64), "wide", 8),
                              ((512, 1032), "outliers", 9), ((272, 520), "normal", 10)]:
        x = rand_bf16(shape, seed + 10 * fmt, kind)
        assert_quant_equal(fmt, x, flags | ops.AXIS_STRIDED, signs=0x3C5A, seed=777,
                           tag=f"strided fmt {fmt} flags {flags} {shape}")


@pytest.mark.parametrize("fmt", FORMATS)
def test_scale_in(fmt):
    x = rand_bf16((96, 512), 9, "outliers")
    for alpha in (1.0, 2.0 ** -7, 0.013, 1e-3):
        assert_quant_equal(fmt, x, ops.SCALE_IN, alpha=alpha, tag=f"scale_in {alpha}")
    # alpha = 0 stores every group as zero
    assert_quant_equal(fmt, x, ops.SCALE_IN, alpha=0.0, tag="scale_in 0")


def test_non_contiguous_rows():
    x = rand_bf16((50, 320), 11, "outliers")
    for fmt in (ops.IF4, ops.IF3, ops.IF6_E2M3):
        assert_quant_equal(fmt, x, 0, ld_pad=24, tag="ld padded")
        assert_quant_equal(fmt, x, ops.RHT | ops.SR, signs=0x1234, seed=5, ld_pad=8, tag="ld padded rht sr")
    # rows of 65 groups with padding: the first 64 groups of a row are read by
    # whole-wavefront loads, the 65th per lane
    xw = rand_bf16((33, 1040), 13, "outliers")
    for fmt in (ops.IF4, ops.NVFP4, ops.IF3, ops.IF6_E3M2, ops.IF4_BS8):
        assert_quant_equal(fmt, xw, 0, ld_pad=8, tag=f"ld padded 65 groups fmt {fmt}")
        assert_quant_equal(fmt, xw, ops.RHT | ops.SR, signs=0x1234, seed=5, ld_pad=56,
                           tag=f"ld padded 65 groups rht sr fmt {fmt}")
        assert_quant_equal(fmt, xw, ops.RHT, signs=0x0FF0, tag=f"ld contiguous 65 groups rht fmt {fmt}")
    # strided axis: ld % 8 == 0 keeps the register path, ld % 8 != 0 the LDS path
    xs = rand_bf16((256, 328), 12, "outliers")
    for fmt in (ops.IF4, ops.NVFP4, ops.IF3):
        for pad in (8, 3):
            assert_quant_equal(fmt, xs, ops.AXIS_STRIDED, ld_pad=pad, tag=f"strided ld +{pad}")
            assert_quant_equal(fmt, xs, ops.AXIS_STRIDED | ops.RHT | ops.SR, signs=0x4321, seed=6,
                               ld_pad=pad, tag=f"strided ld +{pad} rht sr")


def test_ties_and_signed_zero():
    """alpha = 1 and a group maximum of 6 make x-bar equal to the input, so
    the values below sit exactly on FP4 and INT rounding boundaries."""
    fp_mid = [0.25, 0.75, 1.25, 1.75, 2.5, 3.5, 5.0]
    rows = []
    for sgn in (1, -1):
        vals = [6.0] + [sgn * m for m in fp_mid] + [sgn * 0.1, -0.0, 0.0, sgn * 1e-3,
                                                    sgn * 5.999, sgn * 4.5, sgn * 0.2, sgn * 3.0]
        rows.append(vals)
    # values whose INT candidate x*7/6 sits at a half-integer in fp32
    int_ties = [(k + 0.5) * 6 / 7 for k in range(7)]
    rows.append([6.0] + int_ties + [-t for t in int_ties] + [0.0])
    # all-zero group, outlier group, tiny group
    rows.append([0.0] * 16)
    rows.append([6.0] + [1e-4] * 15)
    rows.append([1e-30] * 16)
    x = workloads.to_bf16(np.array(rows))
    for fmt in FORMATS:
        assert_quant_equal(fmt, x, ops.SCALE_IN, alpha=1.0, tag=f"ties fmt {fmt}")
        assert_quant_equal(fmt, x, 0, tag=f"ties auto fmt {fmt}")


def _magnitude_blocks(shape, seed, exps):
    """N(0,1) values whose 1024-value blocks (64 groups along a row-major
    row, one wavefront's share) are scaled by 2^e for e cycling over exps."""
    rng = np.random.default_rng(seed)
    x = rng.standard_normal(shape).reshape(-1, 1024)
    x *= np.exp2(np.array(exps, dtype=np.float64)[np.arange(x.shape[0]) % len(exps)])[:, None]
    return workloads.to_bf16(x.reshape(shape))


@pytest.mark.parametrize("fmt", FORMATS)
def test_sr_scale_quotient_ranges(fmt):
    """The stochastic-rounding quantizers compute amax / (alpha M) by a
    correction of amax * RN(1/(alpha M)) when every lane of a wavefront has
    amax >= 2^-100 and alpha M is normal with a normal reciprocal, and by
    the division otherwise; 1/(alpha Delta) skips its range test when
    alpha * 448 <= 2^126.  Tiny groups (below 2^-100, down to bf16
    subnormals) next to ordinary ones, tiny tensors, and supplied alphas on
    either side of each range limit, against the oracle bit for bit.  (Block
    magnitudes stay below 2^122 so that the RHT's sums of 16 stay finite.)"""
    shape = (256, 1024)  # rows % 256 == 0: the strided 4-bit register path too
    cases = [
        (_magnitude_blocks(shape, 31, [0, -105, -20, -128]), None, "mixed waves"),
        (_magnitude_blocks(shape, 32, [-98, -101, -110, -131]), None, "tiny tensor"),
        (_magnitude_blocks(shape, 33, [0, -3]), 2.0 ** -130, "alpha*M below 2^-125"),
        (_magnitude_blocks(shape, 34, [110, 116]), 2.0 ** 100, "alpha 2^100"),
        (_magnitude_blocks(shape, 35, [118, 121]), 2.0 ** 120, "alpha*448 above 2^126"),
        (_magnitude_blocks(shape, 36, [118, 121]), 2.0 ** 124, "alpha*M above 2^125"),
    ]
    for x, alpha, tag in cases:
        for flags in (ops.SR, ops.SR | ops.RHT | ops.MARGIN_16_17, ops.SR | ops.SR_RTN_TYPE):
            f = flags | (ops.SCALE_IN if alpha is not None else 0)
            assert_quant_equal(fmt, x, f, signs=0x5AC3, seed=99, alpha=alpha,
                               tag=f"fmt {fmt} {tag} flags {f}")
            assert_quant_equal(fmt, x, f | ops.AXIS_STRIDED, signs=0x5AC3, seed=98, alpha=alpha,
                               tag=f"strided fmt {fmt} {tag} flags {f}")


def _bf16_neighbours(v):
    """The bf16 values one step below and above each positive bf16 value v."""
    b = O.bf16_bits(np.asarray(v, dtype=np.float32)).astype(np.int64)
    return (O.bf16_to_f32((b - 1).astype(np.uint16)).astype(np.float64),
            O.bf16_to_f32((b + 1).astype(np.uint16)).astype(np.float64))


def test_every_scale_code_and_tie():
    """With alpha supplied as fp32(1/M), fp32(alpha * M) is exactly 1, so the
    scale quotient of Eq. 2 equals the group maximum.  Group maxima at every
    E4M3 value, at every midpoint between neighbouring codes (a tie, which
    goes to the even code), one bf16 step either side of each midpoint, at
    2^-10 (rounds to the zero scale) and above 448 (saturates) exercise every
    scale code and every rounding boundary between codes."""
    vals = np.array([O.e4m3_value(c) for c in range(127)], dtype=np.float64)
    mids = (vals[:-1] + vals[1:]) / 2
    lo, hi = _bf16_neighbours(mids)
    maxima = np.concatenate([vals[1:], mids, lo, hi, [2.0 ** -10, 448.0, 460.0, 464.0, 500.0, 3.0e4]])
    ng = 16 * int(np.ceil(len(maxima) / 16))
    maxima = np.concatenate([maxima, np.full(ng - len(maxima), 1.0)])
    rng = np.random.default_rng(77)
    g = maxima[:, None] * rng.uniform(-1, 1, (ng, 16))
    g[:, 0] = maxima
    g = g[rng.permutation(ng)]
    for j in range(ng):  # the maximum in a different place in every group
        g[j] = np.roll(g[j], j % 16)
    x = workloads.to_bf16(g.reshape(ng // 16, 256))
    assert np.all(np.abs(bits(x).view(np.uint16) & 0x7FFF) <= 0x7F80)
    targets = {ops.IF3: 4.0, ops.IF6_E2M3: 7.5, ops.IF6_E3M2: 28.0, ops.NVINT4: 7.0, ops.IF3_BS8: 4.0}
    for fmt in FORMATS:
        m = targets.get(fmt, 6.0)
        alpha = float(np.float32(1.0) / np.float32(m))
        assert np.float32(alpha) * np.float32(m) == np.float32(1.0)
        _, (_, osc, _) = assert_quant_equal(fmt, x, ops.SCALE_IN, alpha=alpha, tag=f"scale codes fmt {fmt}")
        if fmt in (ops.IF4, ops.NVFP4):
            assert len(np.unique(osc & 0x7F)) == 127  # every code, 0 included
        assert_quant_equal(fmt, x, ops.SCALE_IN | ops.SR, alpha=alpha, seed=3, tag=f"scale codes sr fmt {fmt}")


@pytest.mark.parametrize("fmt", [ops.IF6_E2M3, ops.IF6_E3M2, ops.IF4, ops.NVFP4, ops.IF3])
def test_fp_grid_midpoints(fmt):
    """alpha = 1 and a group maximum of M_FP make the scale 1, so x-bar is the
    input itself: every midpoint between neighbouring FP grid values (a tie,
    to the even code), one bf16 step either side of it, the grid values and
    values beyond the maximum, in both signs, at every position of a group."""
    grid = O.fp_grid(fmt).astype(np.float64)
    fmax = float(grid.max())
    mids = (grid[:-1] + grid[1:]) / 2
    lo, hi = _bf16_neighbours(mids[mids > 0])
    vals = np.concatenate([grid, mids, lo, hi, [fmax * 1.01, fmax * 1.5]])
    vals = np.concatenate([vals, -vals])
    n = 15 * int(np.ceil(len(vals) / 15))
    vals = np.concatenate([vals, np.zeros(n - len(vals))])
    rows = []
    for k, chunk in enumerate(vals.reshape(-1, 15)):
        g = np.insert(chunk, k % 16, fmax)   # the group maximum M_FP, anywhere in the group
        rows.append(g)
    x = workloads.to_bf16(np.array(rows))  # one group per row
    assert_quant_equal(fmt, x, ops.SCALE_IN, alpha=1.0, tag=f"fp grid midpoints fmt {fmt}")


def test_nvint4_and_four_six_boundaries():
    """NVINT4 with alpha = 1 and group maximum 7 (Delta = 1): half-integers
    are exact rounding ties.  4/6: a group exact only when scaled to 4, a
    group exact both ways (tie keeps 6), and, at alpha = 2^-120, a group
    whose scaling to 6 falls below FLT_MIN while the scaling to 4 does not."""
    halves = [0.5 + k for k in range(7)]
    rows = [[7.0] + halves + [-h for h in halves] + [7.49],
            [7.0] + [-7.0, 6.5, -6.5, 0.25, -0.25, 0.75, -0.75, 3.5, -3.5, 0.0, -0.0, 1e-3, 2.4999, 2.5001, 5.0]]
    x = workloads.to_bf16(np.array(rows))
    assert_quant_equal(ops.NVINT4, x, ops.SCALE_IN, alpha=1.0, tag="nvint4 ties")
    assert_quant_equal(ops.NVINT4, x, ops.SCALE_IN | ops.MARGIN_16_17, alpha=1.0, tag="nvint4 margin")
    rows = [[4.0, -3.0, 2.0, 1.0, 0.5, -1.5] + [0.0] * 10,
            [3.0, -3.0] * 8,
            [6.0, 4.5, 3.0, -2.25, 0.75, 1.5, 0.375] + [0.0] * 9,
            [2.0 ** -124 * 1.25, 2.0 ** -126, -2.0 ** -125] + [0.0] * 13]
    x = workloads.to_bf16(np.array(rows))
    assert_quant_equal(ops.NVFP4_46, x, ops.SCALE_IN, alpha=1.0, tag="4/6 exact")
    oc, osc, _ = O.quantize(bits(x), ops.NVFP4_46, O.SCALE_IN, tensor_scale=1.0)
    assert O.e4m3_value(osc[0, 0]) == 1.0 and O.e4m3_value(osc[1, 0]) == 0.5
    assert_quant_equal(ops.NVFP4_46, x, ops.SCALE_IN, alpha=2.0 ** -120, tag="4/6 tiny alpha")
    oc, osc, _ = O.quantize(bits(x), ops.NVFP4_46, O.SCALE_IN, tensor_scale=2.0 ** -120)
    assert O.e4m3_value(osc[3, 0]) == 1.25 * 2.0 ** -6  # the scaling to 4
    for flags in (ops.SR, ops.SR | ops.SR_RTN_TYPE, ops.SR | ops.MARGIN_16_17):
        assert_quant_equal(ops.NVFP4_46, x, ops.SCALE_IN | flags, alpha=1.0, seed=3,
                           tag=f"4/6 flags {flags}")


def test_zero_and_empty():
    z = torch.zeros((32, 64), dtype=torch.bfloat16)
    for fmt in FORMATS:
        assert_quant_equal(fmt, z, 0, tag="zero")
    p, c, s, a = gpu_quantize(ops.IF4, torch.zeros((0, 64), dtype=torch.bfloat16))
    assert a == 0.0 and c.size == 0 and s.size == 0


@pytest.mark.parametrize("kind", ["quant_sweep", "fwd_mlp", "wgrad", "bitwidth"])
def test_workload_distributions_small(kind):
    """The measured workloads' distributions at 1/16 of each dimension."""
    w = workloads.small_like(kind)
    if kind == "quant_sweep":
        x = w.tensors["X"]
        for fmt in (ops.IF4, ops.NVFP4):
            assert_quant_equal(fmt, x, 0, tag="sweep")
            assert_quant_equal(fmt, x, ops.RHT, signs=w.info["rht_signs"], tag="sweep rht")
    elif kind == "fwd_mlp":
        assert_quant_equal(ops.IF4, w.tensors["A"], tag="acts")
        assert_quant_equal(ops.IF4, w.tensors["W"], tag="weights")
    elif kind == "wgrad":
        fl = ops.AXIS_STRIDED | ops.RHT | ops.SR | ops.MARGIN_16_17
        assert_quant_equal(ops.IF4, w.tensors["dY"], fl, w.info["rht_signs"], w.info["sr_seed_dY"], tag="dY")
        assert_quant_equal(ops.IF4, w.tensors["X"], fl, w.info["rht_signs"], w.info["sr_seed_X"], tag="X")
    else:
        for fmt in FORMATS:
            assert_quant_equal(fmt, w.tensors["A"], tag=f"bitwidth {fmt}")


@pytest.mark.parametrize("fmt", FORMATS)
@pytest.mark.parametrize("dtype", [ops.F32, ops.BF16])
def test_dequantize_bit_exact(fmt, dtype):
    x = rand_bf16((70, 640), 21 + fmt, "outliers")
    for flags in (0, ops.RHT | ops.SR):
        p, (oc, osc, oa) = assert_quant_equal(fmt, x, flags, signs=0x0F0F, seed=3, tag="dq src")
        out = ops.ifx_dequantize(p, dtype).cpu()
        ref = O.dequantize(oc, osc, oa, fmt)
        if dtype == ops.F32:
            got = out.numpy()
            np.testing.assert_array_equal(got.view(np.uint32), ref.view(np.uint32))
        else:
            got = out.view(torch.int16).numpy().view(np.uint16)
            np.testing.assert_array_equal(got, O.bf16_bits(ref))


ADAPTIVE_FORMATS = (ops.IF4, ops.IF3, ops.IF6_E2M3, ops.IF6_E3M2, ops.IF4_BS8, ops.IF3_BS8)


@pytest.mark.parametrize("fmt", FORMATS)
def test_dequantize_every_code_and_scale_byte(fmt):
    """Packed data written directly: random code bits (every code value),
    every finite scale byte (with the indicator bit for the adaptive
    formats), and tensor scales that push the products into fp32 subnormals
    and near the top of the range; fp32 and bf16 outputs bit for bit."""
    rng = np.random.default_rng(120 + fmt)
    rows, cols = 96, 1024
    g = ops.GSIZE[fmt]
    codes = rng.integers(0, 256, (rows, cols * ops.BITS[fmt] // 8), dtype=np.uint8)
    top = 256 if fmt in ADAPTIVE_FORMATS else 128
    vals = np.array([b for b in range(top) if (b & 0x7F) != 0x7F], dtype=np.uint8)
    scales = vals[np.arange(rows * cols // g) % len(vals)].reshape(rows, cols // g)
    for alpha in (1.0, 2.0 ** -120, 3.7e5):
        ts = torch.tensor([alpha], dtype=torch.float32, device="cuda")
        p = ops.Packed(fmt, torch.from_numpy(codes).cuda(), torch.from_numpy(scales).cuda(), ts, rows, cols)
        ref = O.dequantize(codes, scales, np.float32(alpha), fmt)
        got = ops.ifx_dequantize(p, ops.F32).cpu().numpy()
        np.testing.assert_array_equal(got.view(np.uint32), ref.view(np.uint32), err_msg=f"fp32 alpha {alpha}")
        got16 = ops.ifx_dequantize(p, ops.BF16).cpu().view(torch.int16).numpy().view(np.uint16)
        np.testing.assert_array_equal(got16, O.bf16_bits(ref), err_msg=f"bf16 alpha {alpha}")


def test_full_size_quant_sweep():
    """8192x8192 t(3) with outlier columns: IF4 and NVFP4, with and without
    the RHT, bit-exact over the whole tensor."""
    w = workloads.quant_sweep()
    x = w.tensors["X"]
    for fmt in (ops.IF4, ops.NVFP4):
        assert_quant_equal(fmt, x, 0, tag="full sweep")
        assert_quant_equal(fmt, x, ops.RHT, signs=w.info["rht_signs"], tag="full sweep rht")


def test_determinism_repeat():
    x = rand_bf16((512, 1024), 31, "outliers")
    p1, c1, s1, a1 = gpu_quantize(ops.IF4, x, ops.RHT | ops.SR, 0x5555, 9)
    p2, c2, s2, a2 = gpu_quantize(ops.IF4, x, ops.RHT | ops.SR, 0x5555, 9)
    assert a1 == a2 and np.array_equal(c1, c2) and np.array_equal(s1, s2)
