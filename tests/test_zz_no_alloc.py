"""GPU test of the allocation-free quantize entry point: through the C ABI,
ifx_quantize_noalloc must give the same codes, scale bytes and tensor scale,
bit for bit, as ifx_quantize with a caller workspace, on two calls in a row
(the second with a smaller input, so the shared scratch still holds the
first call's partial maxima)."""
import ctypes as C

import numpy as np
import pytest
import torch

from paper_2603_28765_amd import ops, workloads

pytestmark = pytest.mark.gpu


def _call_noalloc(fmt, x, flags, signs, seed, out):
    L = ops.lib()
    st = L.ifx_quantize_noalloc(fmt, x.data_ptr(), x.shape[0], x.shape[1], x.stride(0), flags, signs,
                                seed, out.codes.data_ptr(), out.scales.data_ptr(),
                                out.tensor_scale.data_ptr(), torch.cuda.current_stream().cuda_stream)
    assert st == 0, L.ifq_status_string(st)


def _empty_like(fmt, R, K):
    return ops.Packed(fmt, torch.empty((R, K * ops.BITS[fmt] // 8), dtype=torch.uint8, device="cuda"),
                      torch.empty((R, K // ops.GSIZE[fmt]), dtype=torch.uint8, device="cuda"),
                      torch.empty(1, dtype=torch.float32, device="cuda"), R, K)


@pytest.mark.parametrize("fmt,flags", [
    (ops.IF4, 0), (ops.NVFP4, ops.RHT), (ops.IF4, ops.AXIS_STRIDED | ops.RHT | ops.SR | ops.MARGIN_16_17),
    (ops.IF6_E2M3, 0), (ops.IF4_BS8, ops.SR)])
def test_noalloc_equals_workspace_entry_point(fmt, flags):
    if not torch.cuda.is_available():
        pytest.fail("GPU test run without a GPU")
    rng = np.random.default_rng(500 + fmt + flags)
    signs, seed = 0x6B2D, 77
    # first call large, second smaller: the scratch keeps the first call's
    # partials and the second must not read them
    for shape, scale in (((4096, 2048), 1.0), ((512, 256), 1e-3)):
        x = workloads.to_bf16(rng.standard_t(3, shape) * scale).cuda()
        ref = ops.ifx_quantize(fmt, x, flags, signs, seed)
        R, K = (shape[1], shape[0]) if flags & ops.AXIS_STRIDED else shape
        out = _empty_like(fmt, R, K)
        out.codes.fill_(0xA5)
        out.scales.fill_(0x5A)
        _call_noalloc(fmt, x, flags, signs, seed, out)
        torch.cuda.synchronize()
        assert float(out.tensor_scale.cpu()[0]) == float(ref.tensor_scale.cpu()[0]), shape
        assert torch.equal(out.scales, ref.scales), shape
        assert torch.equal(out.codes, ref.codes), shape
        # the binding's wrapper goes through the same entry point
        again = ops.ifx_quantize_noalloc(fmt, x, flags, signs, seed)
        torch.cuda.synchronize()
        assert torch.equal(again.codes, ref.codes) and torch.equal(again.scales, ref.scales)


def test_noalloc_scale_in_and_empty():
    x = workloads.to_bf16(np.random.default_rng(3).standard_normal((256, 512))).cuda()
    ts = torch.tensor([0.004], dtype=torch.float32, device="cuda")
    ref = ops.ifx_quantize(ops.IF4, x, ops.SCALE_IN, tensor_scale=ts)
    got = ops.ifx_quantize_noalloc(ops.IF4, x, ops.SCALE_IN, tensor_scale=ts.clone())
    torch.cuda.synchronize()
    assert torch.equal(got.codes, ref.codes) and torch.equal(got.scales, ref.scales)
    e = ops.ifx_quantize_noalloc(ops.IF4, torch.zeros((0, 64), dtype=torch.bfloat16, device="cuda"))
    torch.cuda.synchronize()
    assert float(e.tensor_scale.cpu()[0]) == 0.0
