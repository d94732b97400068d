"""Thin Python binding of libifq.so (the C ABI in include/ifq.h).

Argument marshalling only: every step of quantization, dequantization and
the GEMM runs in the HIP kernels of libifq.so.  PyTorch provides device
memory and the current HIP stream.  There is no fallback: if the library is
not built, or a tensor is not on a GPU, these functions raise.

Function names match the C entry points (if4_quantize, nvfp4_gemm, ...).
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libifq.so")

IF4, NVFP4, IF3, IF6_E2M3, IF6_E3M2, NVINT4, NVFP4_46, IF4_BS8, IF3_BS8, NVFP4_BS8 = range(10)
FORMAT_NAMES = {IF4: "if4", NVFP4: "nvfp4", IF3: "if3", IF6_E2M3: "if6_e2m3", IF6_E3M2: "if6_e3m2",
                NVINT4: "nvint4", NVFP4_46: "nvfp4_46", IF4_BS8: "if4_bs8", IF3_BS8: "if3_bs8",
                NVFP4_BS8: "nvfp4_bs8"}
BITS = {IF4: 4, NVFP4: 4, IF3: 3, IF6_E2M3: 6, IF6_E3M2: 6, NVINT4: 4, NVFP4_46: 4, IF4_BS8: 4,
        IF3_BS8: 3, NVFP4_BS8: 4}
# values per scale byte
GSIZE = {f: (8 if f in (IF4_BS8, IF3_BS8, NVFP4_BS8) else 16) for f in BITS}

RHT, SR, MARGIN_16_17, SCALE_IN, AXIS_STRIDED, SR_RTN_TYPE = 1, 2, 4, 8, 16, 32
F32, BF16 = 0, 1

STATUS = {0: "ok", -1: "invalid argument", -2: "invalid shape", -3: "misaligned",
          -4: "unsupported", -5: "HIP launch failed", -6: "workspace too small"}


class IfqError(RuntimeError):
    def __init__(self, fn: str, status: int):
        super().__init__(f"{fn} failed: {STATUS.get(status, status)} ({status})")
        self.status = status


_lib = None

_QUANT_ARGS = [C.c_void_p, C.c_int64, C.c_int64, C.c_int64, C.c_uint32, C.c_uint32, C.c_uint64,
               C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_size_t, C.c_void_p]
_DEQ_ARGS = [C.c_void_p, C.c_void_p, C.c_void_p, C.c_int64, C.c_int64, C.c_void_p, C.c_int,
             C.c_void_p]
_GEMM_ARGS = [C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_int64,
              C.c_int64, C.c_int64, C.c_void_p, C.c_int64, C.c_int, C.c_void_p]


def lib() -> C.CDLL:
    """Load libifq.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -c 'import __graft_entry__ as g; g.build()'`")
        L = C.CDLL(LIB_PATH)
        for name in ("if4_quantize", "nvfp4_quantize"):
            getattr(L, name).argtypes = _QUANT_ARGS
        L.ifx_quantize.argtypes = [C.c_int] + _QUANT_ARGS
        L.ifx_quantize_noalloc.argtypes = [C.c_int] + _QUANT_ARGS[:10] + [C.c_void_p]
        for name in ("if4_dequantize", "nvfp4_dequantize"):
            getattr(L, name).argtypes = _DEQ_ARGS
        L.ifx_dequantize.argtypes = [C.c_int] + _DEQ_ARGS
        for name in ("if4_gemm", "nvfp4_gemm"):
            getattr(L, name).argtypes = _GEMM_ARGS
        L.ifx_gemm.argtypes = [C.c_int] + _GEMM_ARGS
        L.ifq_quantize_workspace_bytes.argtypes = [C.c_int, C.c_int64, C.c_int64, C.c_uint32]
        L.ifq_quantize_workspace_bytes.restype = C.c_size_t
        L.ifq_codes_bytes.argtypes = [C.c_int, C.c_int64, C.c_int64]
        L.ifq_codes_bytes.restype = C.c_size_t
        L.ifq_scales_bytes.argtypes = [C.c_int, C.c_int64, C.c_int64]
        L.ifq_scales_bytes.restype = C.c_size_t
        L.ifx_quantize_dual.argtypes = [C.c_int, C.c_void_p, C.c_int64, C.c_int64, C.c_int64,
                                         C.c_uint32, C.c_uint32, C.c_uint32, C.c_uint64, C.c_uint64,
                                         C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p, C.c_void_p,
                                         C.c_void_p, C.c_void_p, C.c_size_t, C.c_void_p]
        L.ifq_quantize_dual_workspace_bytes.argtypes = [C.c_int, C.c_int64, C.c_int64, C.c_uint32,
                                                        C.c_uint32]
        L.ifq_quantize_dual_workspace_bytes.restype = C.c_size_t
        L.ifq_group_size.argtypes = [C.c_int]
        L.ifq_group_size.restype = C.c_int
        L.ifq_status_string.argtypes = [C.c_int]
        L.ifq_status_string.restype = C.c_char_p
        L.ifq_abi_version.restype = C.c_int
        _lib = L
    return _lib


def _check(fn: str, status: int):
    if status != 0:
        raise IfqError(fn, status)


def _stream(t: torch.Tensor) -> int:
    return torch.cuda.current_stream(t.device).cuda_stream


def _require_gpu(*ts: torch.Tensor):
    for t in ts:
        if not t.is_cuda:
            raise ValueError("libifq operates on GPU tensors only")


def _require_buffer(name: str, t: torch.Tensor, shape, dtype, device):
    """The C ABI receives bare pointers, so every buffer's shape, dtype,
    device and layout is checked here before a launch: a short or strided
    buffer would otherwise be written past its end."""
    if not isinstance(t, torch.Tensor):
        raise ValueError(f"{name} must be a tensor")
    if t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")
    if t.dtype != dtype:
        raise ValueError(f"{name} has dtype {t.dtype}, expected {dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} has shape {tuple(t.shape)}, expected {tuple(shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _require_packed(name: str, p: "Packed", device=None):
    """A Packed operand must hold exactly the buffers its format and logical
    shape [rows, cols] imply."""
    if p.fmt not in BITS:
        raise ValueError(f"{name}: unknown format {p.fmt}")
    if p.cols % 16:
        raise ValueError(f"{name}: K = {p.cols} is not a multiple of 16")
    dev = p.codes.device if device is None else device
    _require_gpu(p.codes)
    _require_buffer(f"{name}.codes", p.codes, (p.rows, p.cols * BITS[p.fmt] // 8), torch.uint8, dev)
    _require_buffer(f"{name}.scales", p.scales, (p.rows, p.cols // GSIZE[p.fmt]), torch.uint8, dev)
    _require_buffer(f"{name}.tensor_scale", p.tensor_scale, (1,), torch.float32, dev)


@dataclass
class Packed:
    """A quantized tensor: codes [R, K*bits/8], scales [R, K/16] (uint8),
    tensor_scale (1 float32), all on the GPU; logical shape [R, K]."""
    fmt: int
    codes: torch.Tensor
    scales: torch.Tensor
    tensor_scale: torch.Tensor
    rows: int
    cols: int


def _quantize(fn: str, fmt: int, x: torch.Tensor, flags: int = 0, rht_signs: int = 0,
              seed: int = 0, tensor_scale: torch.Tensor | None = None,
              out: Packed | None = None, workspace: torch.Tensor | None = None) -> Packed:
    _require_gpu(x)
    if x.dtype != torch.bfloat16 or x.dim() != 2 or x.stride(1) != 1:
        raise ValueError("x must be a 2-D bf16 GPU tensor with unit column stride")
    rows, cols = x.shape
    R, K = (cols, rows) if flags & AXIS_STRIDED else (rows, cols)
    dev = x.device
    if fmt not in BITS:
        raise ValueError(f"unknown format {fmt}")
    if out is None:
        codes = torch.empty((R, K * BITS[fmt] // 8), dtype=torch.uint8, device=dev)
        scales = torch.empty((R, K // GSIZE[fmt]), dtype=torch.uint8, device=dev)
        ts = torch.empty(1, dtype=torch.float32, device=dev) if tensor_scale is None else tensor_scale
        out = Packed(fmt, codes, scales, ts, R, K)
    else:
        if (out.fmt, out.rows, out.cols) != (fmt, R, K):
            raise ValueError(f"out describes format {out.fmt} [{out.rows}, {out.cols}], the call "
                             f"writes format {fmt} [{R}, {K}]")
        if tensor_scale is not None:
            out.tensor_scale = tensor_scale
    if flags & SCALE_IN and tensor_scale is None:
        raise ValueError("SCALE_IN needs tensor_scale")
    if K % 16 == 0:  # other shapes are rejected by the library itself
        _require_packed("out", out, dev)
    L = lib()
    wsb = 0 if fn == "ifx_quantize_noalloc" else L.ifq_quantize_workspace_bytes(fmt, rows, cols, flags)
    if wsb and workspace is None:
        workspace = torch.empty(max(wsb, 256), dtype=torch.uint8, device=dev)
    ws_ptr = workspace.data_ptr() if workspace is not None else None
    ws_len = workspace.numel() if workspace is not None else 0
    args = (x.data_ptr(), rows, cols, x.stride(0), flags, rht_signs, seed, out.codes.data_ptr(),
            out.scales.data_ptr(), out.tensor_scale.data_ptr(), ws_ptr, ws_len, _stream(x))
    if fn == "ifx_quantize_noalloc":
        _check(fn, L.ifx_quantize_noalloc(fmt, *args[:10], args[12]))
    elif fn == "ifx_quantize":
        _check(fn, L.ifx_quantize(fmt, *args))
    else:
        _check(fn, getattr(L, fn)(*args))
    return out


def if4_quantize(x, flags=0, rht_signs=0, seed=0, tensor_scale=None, out=None, workspace=None):
    return _quantize("if4_quantize", IF4, x, flags, rht_signs, seed, tensor_scale, out, workspace)


def nvfp4_quantize(x, flags=0, rht_signs=0, seed=0, tensor_scale=None, out=None, workspace=None):
    return _quantize("nvfp4_quantize", NVFP4, x, flags, rht_signs, seed, tensor_scale, out,
                     workspace)


def ifx_quantize(fmt, x, flags=0, rht_signs=0, seed=0, tensor_scale=None, out=None,
                 workspace=None):
    return _quantize("ifx_quantize", fmt, x, flags, rht_signs, seed, tensor_scale, out, workspace)


def ifx_quantize_noalloc(fmt, x, flags=0, rht_signs=0, seed=0, tensor_scale=None, out=None):
    """ifx_quantize through the entry point that allocates nothing: the
    library keeps its tensor-max partials in its own device scratch.  Pass
    `out` (and `tensor_scale`) to keep this call free of allocations on the
    Python side as well."""
    return _quantize("ifx_quantize_noalloc", fmt, x, flags, rht_signs, seed, tensor_scale, out)


def _packed_for(fmt: int, R: int, K: int, dev, tensor_scale=None) -> Packed:
    codes = torch.empty((R, K * BITS[fmt] // 8), dtype=torch.uint8, device=dev)
    scales = torch.empty((R, K // GSIZE[fmt]), dtype=torch.uint8, device=dev)
    ts = torch.empty(1, dtype=torch.float32, device=dev) if tensor_scale is None else tensor_scale
    return Packed(fmt, codes, scales, ts, R, K)


def ifx_quantize_dual(fmt, x, row_flags=0, col_flags=0, rht_signs=0, row_seed=0, col_seed=0,
                      row_tensor_scale=None, col_tensor_scale=None, out_row=None, out_col=None,
                      workspace=None):
    """Both layouts of x from one read: (row-wise Packed [rows, cols],
    strided Packed describing x^T [cols, rows]); see ifx_quantize_dual in
    include/ifq.h."""
    _require_gpu(x)
    if x.dtype != torch.bfloat16 or x.dim() != 2 or x.stride(1) != 1:
        raise ValueError("x must be a 2-D bf16 GPU tensor with unit column stride")
    rows, cols = x.shape
    dev = x.device
    if fmt not in BITS:
        raise ValueError(f"unknown format {fmt}")
    if out_row is None:
        out_row = _packed_for(fmt, rows, cols, dev, row_tensor_scale)
    elif row_tensor_scale is not None:
        out_row.tensor_scale = row_tensor_scale
    if out_col is None:
        out_col = _packed_for(fmt, cols, rows, dev, col_tensor_scale)
    elif col_tensor_scale is not None:
        out_col.tensor_scale = col_tensor_scale
    if (out_row.fmt, out_row.rows, out_row.cols) != (fmt, rows, cols) or \
            (out_col.fmt, out_col.rows, out_col.cols) != (fmt, cols, rows):
        raise ValueError("out_row / out_col do not describe this format and shape")
    if rows % 16 == 0 and cols % 16 == 0:  # other shapes are rejected by the library itself
        _require_packed("out_row", out_row, dev)
        _require_packed("out_col", out_col, dev)
    L = lib()
    wsb = L.ifq_quantize_dual_workspace_bytes(fmt, rows, cols, row_flags, col_flags)
    if wsb and workspace is None:
        workspace = torch.empty(wsb, dtype=torch.uint8, device=dev)
    ws_ptr = workspace.data_ptr() if workspace is not None else None
    ws_len = workspace.numel() if workspace is not None else 0
    _check("ifx_quantize_dual", L.ifx_quantize_dual(
        fmt, x.data_ptr(), rows, cols, x.stride(0), row_flags, col_flags, rht_signs, row_seed,
        col_seed, out_row.codes.data_ptr(), out_row.scales.data_ptr(),
        out_row.tensor_scale.data_ptr(), out_col.codes.data_ptr(), out_col.scales.data_ptr(),
        out_col.tensor_scale.data_ptr(), ws_ptr, ws_len, _stream(x)))
    return out_row, out_col


def _dequantize(fn: str, p: Packed, out_dtype: int = F32, out: torch.Tensor | None = None,
                fixed_fmt: int | None = None):
    _require_gpu(p.codes, p.scales, p.tensor_scale)
    if fixed_fmt is not None and p.fmt != fixed_fmt:
        raise ValueError(f"{fn} takes {FORMAT_NAMES[fixed_fmt]} data, got format {p.fmt}")
    if out_dtype not in (F32, BF16):
        raise ValueError(f"unknown output dtype {out_dtype}")
    _require_packed("p", p)
    odt = torch.bfloat16 if out_dtype == BF16 else torch.float32
    if out is None:
        out = torch.empty((p.rows, p.cols), device=p.codes.device, dtype=odt)
    _require_buffer("out", out, (p.rows, p.cols), odt, p.codes.device)
    L = lib()
    args = (p.codes.data_ptr(), p.scales.data_ptr(), p.tensor_scale.data_ptr(), p.rows, p.cols,
            out.data_ptr(), out_dtype, _stream(p.codes))
    if fn == "ifx_dequantize":
        _check(fn, L.ifx_dequantize(p.fmt, *args))
    else:
        _check(fn, getattr(L, fn)(*args))
    return out


def if4_dequantize(p: Packed, out_dtype=F32, out=None):
    return _dequantize("if4_dequantize", p, out_dtype, out, IF4)


def nvfp4_dequantize(p: Packed, out_dtype=F32, out=None):
    return _dequantize("nvfp4_dequantize", p, out_dtype, out, NVFP4)


def ifx_dequantize(p: Packed, out_dtype=F32, out=None):
    return _dequantize("ifx_dequantize", p, out_dtype, out)


def _gemm(fn: str, a: Packed, b: Packed, out_dtype: int = F32, out: torch.Tensor | None = None,
          fixed_fmt: int | None = None):
    _require_gpu(a.codes, b.codes)
    if a.fmt != b.fmt:
        raise ValueError(f"A is format {a.fmt} and B format {b.fmt}: one GEMM takes one format")
    if fixed_fmt is not None and a.fmt != fixed_fmt:
        raise ValueError(f"{fn} takes {FORMAT_NAMES[fixed_fmt]} operands, got format {a.fmt}")
    if a.cols != b.cols:
        raise ValueError("A and B must share the grouped axis K")
    if out_dtype not in (F32, BF16):
        raise ValueError(f"unknown output dtype {out_dtype}")
    dev = a.codes.device
    _require_packed("A", a, dev)
    _require_packed("B", b, dev)
    M, N, K = a.rows, b.rows, a.cols
    odt = torch.bfloat16 if out_dtype == BF16 else torch.float32
    if out is None:
        out = torch.empty((M, N), device=dev, dtype=odt)
    if out.device != dev or out.dtype != odt or tuple(out.shape) != (M, N) or \
            (M > 0 and N > 0 and (out.stride(1) != 1 or out.stride(0) < N)):
        raise ValueError(f"out must be a {odt} [{M}, {N}] tensor on {dev} with unit column stride "
                         f"and row stride >= N")
    L = lib()
    args = (a.codes.data_ptr(), a.scales.data_ptr(), a.tensor_scale.data_ptr(), b.codes.data_ptr(),
            b.scales.data_ptr(), b.tensor_scale.data_ptr(), M, N, K, out.data_ptr(), out.stride(0),
            out_dtype, _stream(a.codes))
    if fn == "ifx_gemm":
        _check(fn, L.ifx_gemm(a.fmt, *args))
    else:
        _check(fn, getattr(L, fn)(*args))
    return out


def if4_gemm(a: Packed, b: Packed, out_dtype=F32, out=None):
    return _gemm("if4_gemm", a, b, out_dtype, out, IF4)


def nvfp4_gemm(a: Packed, b: Packed, out_dtype=F32, out=None):
    return _gemm("nvfp4_gemm", a, b, out_dtype, out, NVFP4)


def ifx_gemm(a: Packed, b: Packed, out_dtype=F32, out=None):
    return _gemm("ifx_gemm", a, b, out_dtype, out)
