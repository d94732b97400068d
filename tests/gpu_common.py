"""Helpers shared by the GPU parity tests: run the HIP path through the
Python binding of the C ABI and the CPU oracle on the same bf16 bits."""
import numpy as np
import pytest
import torch

import oracle as O
from paper_2603_28765_amd import ops

FORMATS = [ops.IF4, ops.NVFP4, ops.IF3, ops.IF6_E2M3, ops.IF6_E3M2, ops.NVINT4, ops.NVFP4_46,
           ops.IF4_BS8, ops.IF3_BS8, ops.NVFP4_BS8]
GEMM_FORMATS = FORMATS


def require_gpu():
    if not torch.cuda.is_available():
        pytest.fail("GPU test run without a GPU")
    ops.lib()  # raises if libifq.so is missing


def bits(x_bf16_cpu: torch.Tensor) -> np.ndarray:
    return x_bf16_cpu.contiguous().view(torch.int16).numpy().view(np.uint16)


def gpu_quantize(fmt, x_cpu, flags=0, signs=0, seed=0, alpha=None, ld_pad=0):
    """Quantize on the GPU; returns numpy (codes, scales, alpha)."""
    if ld_pad:
        big = torch.zeros((x_cpu.shape[0], x_cpu.shape[1] + ld_pad), dtype=torch.bfloat16)
        big[:, : x_cpu.shape[1]] = x_cpu
        xg = big.cuda()[:, : x_cpu.shape[1]]
    else:
        xg = x_cpu.cuda()
    ts = None
    if alpha is not None:
        ts = torch.tensor([alpha], dtype=torch.float32, device="cuda")
    p = ops.ifx_quantize(fmt, xg, flags, signs, seed, ts)
    torch.cuda.synchronize()
    return p, p.codes.cpu().numpy(), p.scales.cpu().numpy(), float(p.tensor_scale.cpu()[0])


def oracle_quantize(fmt, x_cpu, flags=0, signs=0, seed=0, alpha=None):
    return O.quantize(bits(x_cpu), fmt, flags, signs, seed, alpha)


def assert_quant_equal(fmt, x_cpu, flags=0, signs=0, seed=0, alpha=None, ld_pad=0, tag=""):
    p, c, s, a = gpu_quantize(fmt, x_cpu, flags, signs, seed, alpha, ld_pad)
    oc, osc, oa = oracle_quantize(fmt, x_cpu, flags, signs, seed, alpha)
    assert a == oa or (np.isnan(a) and np.isnan(oa)), (tag, "alpha", a, oa)
    assert s.shape == osc.shape and c.shape == oc.shape, tag
    if not np.array_equal(s, osc):
        bad = np.argwhere(s != osc)
        raise AssertionError(f"{tag}: {len(bad)} scale bytes differ, first at {bad[0]}: "
                             f"gpu {s[tuple(bad[0])]:#x} oracle {osc[tuple(bad[0])]:#x}")
    if not np.array_equal(c, oc):
        bad = np.argwhere(c != oc)
        raise AssertionError(f"{tag}: {len(bad)} code bytes differ, first at {bad[0]}: "
                             f"gpu {c[tuple(bad[0])]:#x} oracle {oc[tuple(bad[0])]:#x}")
    return p, (oc, osc, oa)


def rel_fro(c, ref):
    c = np.asarray(c, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = np.linalg.norm(ref)
    return np.linalg.norm(c - ref) / (den if den > 0 else 1.0)


def bf16_round(a: np.ndarray) -> np.ndarray:
    return O.bf16_to_f32(O.bf16_bits(np.asarray(a, dtype=np.float32))).astype(np.float64)
