"""CPU oracle for the adaptive block-scaled formats (IF3, IF4, IF6) and the
comparison formats NVFP4, NVINT4 and NVFP4 with 4/6.

TEST INFRASTRUCTURE.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  The product
path (``paper_2603_28765_amd``) never imports, links or calls it, and the two
share no code: this package wraps the scalar C oracle in ``ifq_oracle.c``
(quantize, dequantize, Philox, RHT) and adds the fp64 GEMM reference.

Array conventions follow the format statement of the paper (Sec. 3):
codes are dense little-endian bit streams per group of 16 (for IF4 the
element 2i sits in the low nibble of byte i), scales are one byte per group
(E4M3 magnitude in bits 0-6, bit 7 set for an INT group) and the FP32 tensor
scale alpha is a Python float.
"""
from __future__ import annotations

import ctypes as C
import numpy as np

from . import build as _build

(FMT_IF4, FMT_NVFP4, FMT_IF3, FMT_IF6_E2M3, FMT_IF6_E3M2, FMT_NVINT4,
 FMT_NVFP4_46, FMT_IF4_BS8, FMT_IF3_BS8, FMT_NVFP4_BS8) = range(10)
FORMATS = {"if4": FMT_IF4, "nvfp4": FMT_NVFP4, "if3": FMT_IF3,
           "if6_e2m3": FMT_IF6_E2M3, "if6_e3m2": FMT_IF6_E3M2, "nvint4": FMT_NVINT4,
           "nvfp4_46": FMT_NVFP4_46, "if4_bs8": FMT_IF4_BS8, "if3_bs8": FMT_IF3_BS8,
           "nvfp4_bs8": FMT_NVFP4_BS8}
BITS = {FMT_IF4: 4, FMT_NVFP4: 4, FMT_IF3: 3, FMT_IF6_E2M3: 6, FMT_IF6_E3M2: 6,
        FMT_NVINT4: 4, FMT_NVFP4_46: 4, FMT_IF4_BS8: 4, FMT_IF3_BS8: 3, FMT_NVFP4_BS8: 4}
# values per group (one scale byte each): block size 8 for the *_BS8 formats (Sec. 5.1, Table 6 in App. D)
GSIZE = {f: (8 if f in (FMT_IF4_BS8, FMT_IF3_BS8, FMT_NVFP4_BS8) else 16) for f in BITS}

RHT, SR, MARGIN, SCALE_IN, STRIDED, SR_RTN_TYPE = 1, 2, 4, 8, 16, 32
GROUP = 16

_lib = None


def lib():
    global _lib
    if _lib is None:
        path = _build.build()
        L = C.CDLL(path)
        u8p = C.POINTER(C.c_uint8)
        u16p = C.POINTER(C.c_uint16)
        u32p = C.POINTER(C.c_uint32)
        f32p = C.POINTER(C.c_float)
        f64p = C.POINTER(C.c_double)
        L.oracle_e4m3_value.argtypes = [C.c_int]
        L.oracle_e4m3_value.restype = C.c_double
        L.oracle_e4m3_encode.argtypes = [C.c_float]
        L.oracle_e4m3_encode.restype = C.c_int
        L.oracle_fp_round_index.argtypes = [C.c_int, C.c_float]
        L.oracle_fp_round_index.restype = C.c_int
        L.oracle_fp_magnitude.argtypes = [C.c_int, C.c_int]
        L.oracle_fp_magnitude.restype = C.c_double
        L.oracle_group_size.argtypes = [C.c_int]
        L.oracle_group_size.restype = C.c_int
        L.oracle_fmt_constants.argtypes = [C.c_int, f32p, C.POINTER(C.c_int), f32p, f32p,
                                           C.POINTER(C.c_int)]
        L.oracle_philox4x32_10.argtypes = [u32p, u32p, u32p]
        L.oracle_sr_bits.argtypes = [C.c_uint64, C.c_uint64, u16p]
        L.oracle_rht16.argtypes = [f32p, C.c_uint32, f32p]
        L.oracle_tensor_scale.argtypes = [C.c_int, C.c_float, C.c_uint32]
        L.oracle_tensor_scale.restype = C.c_float
        L.oracle_quantize_group.argtypes = [C.c_int, f32p, C.c_float, C.c_uint32, u16p, u8p,
                                            u8p, f32p, f32p]
        L.oracle_pack_group.argtypes = [C.c_int, u8p, u8p]
        L.oracle_unpack_group.argtypes = [C.c_int, u8p, u8p]
        L.oracle_quantize.argtypes = [C.c_int, u16p, C.c_int64, C.c_int64, C.c_int64,
                                      C.c_uint32, C.c_uint32, C.c_uint64, u8p, u8p, f32p]
        L.oracle_quantize.restype = C.c_int
        L.oracle_dequantize.argtypes = [C.c_int, u8p, u8p, C.c_float, C.c_int64, C.c_int64,
                                        f32p]
        L.oracle_dequantize.restype = C.c_int
        L.oracle_dequantize_f64.argtypes = [C.c_int, u8p, u8p, C.c_float, C.c_int64,
                                            C.c_int64, f64p]
        L.oracle_dequantize_f64.restype = C.c_int
        _lib = L
    return _lib


def _ptr(a: np.ndarray, ctype):
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(C.POINTER(ctype))


# ----------------------------------------------------------------- codecs --

def e4m3_value(code: int) -> float:
    """Value of a non-negative E4M3 code (bits 0-6)."""
    return lib().oracle_e4m3_value(int(code))


def e4m3_encode(x: float) -> int:
    """Nearest E4M3 code to x >= 0 (ties to even code, saturating at 448)."""
    return lib().oracle_e4m3_encode(float(x))


def fp_magnitude(fmt: int, idx: int) -> float:
    return lib().oracle_fp_magnitude(fmt, idx)


def fp_grid(fmt: int) -> np.ndarray:
    n = 1 << (BITS[fmt] - 1)
    return np.array([fp_magnitude(fmt, i) for i in range(n)])


def fp_round_index(fmt: int, m: float) -> int:
    return lib().oracle_fp_round_index(fmt, float(m))


def fmt_constants(fmt: int) -> dict:
    fp_max, c_up, k_dn = C.c_float(), C.c_float(), C.c_float()
    int_max, bits = C.c_int(), C.c_int()
    lib().oracle_fmt_constants(fmt, C.byref(fp_max), C.byref(int_max), C.byref(c_up),
                               C.byref(k_dn), C.byref(bits))
    return {"fp_max": fp_max.value, "int_max": int_max.value, "c_up": c_up.value,
            "k_dn": k_dn.value, "bits": bits.value}


def tensor_scale(fmt: int, amax: float, flags: int = 0) -> float:
    return lib().oracle_tensor_scale(fmt, float(amax), flags)


# ---------------------------------------------------------- RNG and RHT --

def philox4x32_10(ctr, key) -> np.ndarray:
    c = np.ascontiguousarray(np.asarray(ctr, dtype=np.uint32))
    k = np.ascontiguousarray(np.asarray(key, dtype=np.uint32))
    out = np.zeros(4, dtype=np.uint32)
    lib().oracle_philox4x32_10(_ptr(c, C.c_uint32), _ptr(k, C.c_uint32), _ptr(out, C.c_uint32))
    return out


def sr_bits(seed: int, group: int) -> np.ndarray:
    out = np.zeros(GROUP, dtype=np.uint16)
    lib().oracle_sr_bits(seed, group, _ptr(out, C.c_uint16))
    return out


def rht16(x, signs: int) -> np.ndarray:
    xv = np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    assert xv.shape == (GROUP,)
    out = np.zeros(GROUP, dtype=np.float32)
    lib().oracle_rht16(_ptr(xv, C.c_float), signs, _ptr(out, C.c_float))
    return out


# ------------------------------------------------------------ one group --

def group_size(fmt: int) -> int:
    return lib().oracle_group_size(fmt)


def quantize_group(v, alpha: float, fmt: int = FMT_IF4, flags: int = 0, h=None):
    """Returns (codes[n] uint8, scale byte, E_FP, E_INT) for one group of
    n = GSIZE[fmt] values (for 4/6: the errors of the scalings to 6 and to 4
    in alpha units)."""
    n = GSIZE[fmt]
    vv = np.zeros(GROUP, dtype=np.float32)
    vin = np.asarray(v, dtype=np.float32)
    assert vin.shape == (n,)
    vv[:n] = vin
    hh = np.zeros(GROUP, dtype=np.uint16)
    if h is not None:
        hin = np.asarray(h, dtype=np.uint16)
        hh[: len(hin)] = hin
    codes = np.zeros(GROUP, dtype=np.uint8)
    sb = np.zeros(1, dtype=np.uint8)
    ef, ei = C.c_float(), C.c_float()
    lib().oracle_quantize_group(fmt, _ptr(vv, C.c_float), float(alpha), flags,
                                _ptr(hh, C.c_uint16), _ptr(codes, C.c_uint8),
                                _ptr(sb, C.c_uint8), C.byref(ef), C.byref(ei))
    return codes[:n], int(sb[0]), ef.value, ei.value


def pack_group(fmt: int, codes) -> np.ndarray:
    c = np.zeros(GROUP, dtype=np.uint8)
    cin = np.asarray(codes, dtype=np.uint8)
    c[: len(cin)] = cin
    out = np.zeros(GSIZE[fmt] * BITS[fmt] // 8, dtype=np.uint8)
    lib().oracle_pack_group(fmt, _ptr(c, C.c_uint8), _ptr(out, C.c_uint8))
    return out


def unpack_group(fmt: int, packed) -> np.ndarray:
    p = np.ascontiguousarray(np.asarray(packed, dtype=np.uint8))
    out = np.zeros(GROUP, dtype=np.uint8)
    lib().oracle_unpack_group(fmt, _ptr(p, C.c_uint8), _ptr(out, C.c_uint8))
    return out[: GSIZE[fmt]]


# --------------------------------------------------------- whole tensors --

def codes_shape(fmt: int, rows: int, cols: int, flags: int = 0):
    out_rows, k = (cols, rows) if flags & STRIDED else (rows, cols)
    return (out_rows, k * BITS[fmt] // 8), (out_rows, k // GSIZE[fmt])


def quantize(x_bf16_bits: np.ndarray, fmt: int = FMT_IF4, flags: int = 0, rht_signs: int = 0,
             seed: int = 0, tensor_scale: float | None = None, ld_x: int | None = None):
    """Quantize a 2-D bf16 matrix given as its uint16 bit patterns.

    Returns (codes, scales, alpha).  With STRIDED in flags the groups run
    along rows and the outputs describe the transposed matrix.
    """
    x = np.ascontiguousarray(x_bf16_bits, dtype=np.uint16)
    assert x.ndim == 2
    rows = x.shape[0]
    cols = x.shape[1] if ld_x is None else int(ld_x)
    if ld_x is not None:
        raise NotImplementedError("pass a contiguous matrix")
    cshape, sshape = codes_shape(fmt, rows, cols, flags)
    codes = np.zeros(cshape, dtype=np.uint8)
    scales = np.zeros(sshape, dtype=np.uint8)
    ts = np.zeros(1, dtype=np.float32)
    if flags & SCALE_IN:
        assert tensor_scale is not None
        ts[0] = tensor_scale
    rc = lib().oracle_quantize(fmt, _ptr(x, C.c_uint16), rows, cols, cols, flags, rht_signs,
                               seed, _ptr(codes, C.c_uint8), _ptr(scales, C.c_uint8),
                               _ptr(ts, C.c_float))
    if rc != 0:
        raise ValueError("oracle_quantize rejected its arguments")
    return codes, scales, float(ts[0])


def dequantize(codes: np.ndarray, scales: np.ndarray, alpha: float, fmt: int = FMT_IF4,
               dtype=np.float32) -> np.ndarray:
    """fp32 dequantization (q * Delta [* M_FP/M_I] * alpha, in that order)."""
    codes = np.ascontiguousarray(codes, dtype=np.uint8)
    scales = np.ascontiguousarray(scales, dtype=np.uint8)
    rows, cols = scales.shape[0], scales.shape[1] * GSIZE[fmt]
    if dtype == np.float64:
        out = np.zeros((rows, cols), dtype=np.float64)
        rc = lib().oracle_dequantize_f64(fmt, _ptr(codes, C.c_uint8), _ptr(scales, C.c_uint8),
                                         float(alpha), rows, cols, _ptr(out, C.c_double))
    else:
        out = np.zeros((rows, cols), dtype=np.float32)
        rc = lib().oracle_dequantize(fmt, _ptr(codes, C.c_uint8), _ptr(scales, C.c_uint8),
                                     float(alpha), rows, cols, _ptr(out, C.c_float))
    if rc != 0:
        raise ValueError("oracle_dequantize rejected its arguments")
    return out


def gemm_ref(a_codes, a_scales, a_alpha, b_codes, b_scales, b_alpha, fmt: int = FMT_IF4):
    """fp64 reference C = A_hat @ B_hat^T of the exactly dequantized operands
    (both packed along K).  numpy's fp64 matmul stands in for the exact sum."""
    A = dequantize(a_codes, a_scales, a_alpha, fmt, dtype=np.float64)
    B = dequantize(b_codes, b_scales, b_alpha, fmt, dtype=np.float64)
    return A @ B.T


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """fp32/fp64 array -> bf16 bit patterns, round to nearest even."""
    f = np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    u = f.view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return rounded.astype(np.uint16)


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)
