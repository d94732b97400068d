"""The C ABI on a machine without a GPU: the library loads, exports every
entry point include/ifq.h declares, and rejects bad arguments on the host
before enqueueing anything (no compute call is made here)."""
import ctypes as C
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ifq.h")

EINVAL, ESHAPE, EALIGN, EUNSUPPORTED, EWORKSPACE = -1, -2, -3, -4, -6


@pytest.fixture(scope="module")
def L():
    from paper_2603_28765_amd import ops
    if not os.path.exists(ops.LIB_PATH):
        pytest.fail("libifq.so not built (run __graft_entry__.build())")
    return ops.lib()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\*?\s+\**(\w+)\s*\(", text, flags=re.M)))


def test_header_declares_the_entry_points():
    names = declared_functions()
    for base in ("quantize", "dequantize", "gemm"):
        for fam in ("if4", "nvfp4", "ifx"):
            assert f"{fam}_{base}" in names
    assert len(names) >= 14


def test_every_declared_symbol_is_exported(L):
    for name in declared_functions():
        assert hasattr(L, name), name


def test_version_and_strings(L):
    assert L.ifq_abi_version() == 2
    assert L.ifq_status_string(0) == b"ok"
    assert L.ifq_status_string(-2) == b"invalid shape"
    assert L.ifq_codes_bytes(0, 256, 256) == 256 * 128
    assert L.ifq_codes_bytes(2, 16, 64) == 16 * 64 * 3 // 8
    assert L.ifq_codes_bytes(3, 16, 64) == 16 * 64 * 6 // 8
    assert L.ifq_scales_bytes(0, 256, 4096) == 256 * 256
    assert L.ifq_scales_bytes(7, 256, 4096) == 256 * 512      # block size 8: one byte per 8 values
    assert L.ifq_scales_bytes(8, 16, 64) == 16 * 8 and L.ifq_scales_bytes(9, 16, 64) == 16 * 8
    assert L.ifq_scales_bytes(10, 16, 64) == 0 and L.ifq_scales_bytes(0, -1, 64) == 0
    assert L.ifq_quantize_workspace_bytes(0, 8192, 8192, 0) >= 4
    assert L.ifq_quantize_workspace_bytes(0, 8192, 8192, 8) == 0
    assert L.ifq_quantize_dual_workspace_bytes(0, 8192, 8192, 0, 8) >= 8
    assert L.ifq_quantize_dual_workspace_bytes(0, 8192, 8192, 8, 8) == 0
    assert "ifx_quantize_dual" in declared_functions()
    assert [L.ifq_group_size(f) for f in range(11)] == [16] * 7 + [8] * 3 + [0]
    assert L.ifq_codes_bytes(7, 16, 64) == 16 * 64 // 2 and L.ifq_codes_bytes(8, 16, 64) == 16 * 64 * 3 // 8


# fake, never dereferenced device addresses: validation fails first
P16 = 0x100000
P_ODD = 0x100001


def q(L, fmt=None, x=P16, rows=32, cols=64, ld=64, flags=0, signs=0, codes=P16, scales=P16,
      ts=P16, ws=P16, wsb=4096):
    args = (x, rows, cols, ld, flags, signs, 0, codes, scales, ts, ws, wsb, None)
    if fmt is None:
        return L.if4_quantize(*args)
    return L.ifx_quantize(fmt, *args)


def test_quantize_validation(L):
    assert q(L, ts=None) == EINVAL
    assert q(L, x=None) == EINVAL
    assert q(L, codes=None) == EINVAL
    assert q(L, flags=1 << 7) == EINVAL
    assert q(L, signs=1 << 16) == EINVAL
    assert q(L, fmt=10) == EINVAL
    assert q(L, fmt=6, cols=40) == ESHAPE
    assert q(L, fmt=7, cols=40, ld=40) == ESHAPE   # block size 8: K still a multiple of 16
    assert q(L, rows=-1) == ESHAPE
    assert q(L, cols=40, ld=40) == ESHAPE                  # K % 16
    assert q(L, rows=40, flags=16) == ESHAPE               # strided: rows % 16
    assert q(L, ld=48) == ESHAPE                           # ld < cols
    assert q(L, rows=1 << 30, cols=1 << 20, ld=1 << 20) == ESHAPE
    assert q(L, x=P_ODD) == EALIGN
    assert q(L, ld=68) == EALIGN                           # row starts not 16-byte aligned
    assert q(L, codes=P16 + 8) == EALIGN
    assert q(L, ws=None) == EWORKSPACE
    assert q(L, wsb=8) == EWORKSPACE


def test_noalloc_quantize_validation(L):
    """The allocation-free entry point checks its arguments like
    ifx_quantize before it touches the device (no workspace argument)."""
    qn = lambda fmt=0, x=P16, rows=32, cols=64, ld=64, flags=0, signs=0, codes=P16, ts=P16: \
        L.ifx_quantize_noalloc(fmt, x, rows, cols, ld, flags, signs, 0, codes, P16, ts, None)
    assert qn(ts=None) == EINVAL
    assert qn(x=None) == EINVAL
    assert qn(fmt=10) == EINVAL
    assert qn(flags=1 << 7) == EINVAL
    assert qn(signs=1 << 16) == EINVAL
    assert qn(cols=40, ld=40) == ESHAPE
    assert qn(rows=40, flags=16) == ESHAPE
    assert qn(ld=48) == ESHAPE
    assert qn(x=P_ODD) == EALIGN
    assert qn(codes=P16 + 8) == EALIGN


def g(L, fmt=None, a=P16, b=P16, M=64, N=64, K=64, c=P16, ldc=64, dtype=0, ts=P16):
    args = (a, P16, ts, b, P16, ts, M, N, K, c, ldc, dtype, None)
    if fmt is None:
        return L.if4_gemm(*args)
    return L.ifx_gemm(fmt, *args)


def test_gemm_validation(L):
    assert g(L, K=40) == ESHAPE
    assert g(L, M=-1) == ESHAPE
    assert g(L, ldc=32) == ESHAPE
    assert g(L, c=None) == EINVAL
    assert g(L, ts=None) == EINVAL
    assert g(L, dtype=5) == EINVAL
    assert g(L, a=P16 + 4) == EALIGN
    assert g(L, fmt=3, K=40) == ESHAPE    # IF6 GEMM is validated like the others
    assert g(L, fmt=4, ldc=32) == ESHAPE
    assert g(L, fmt=5, K=40) == ESHAPE    # NVINT4 and NVFP4 with 4/6 likewise
    assert g(L, fmt=6, ldc=32) == ESHAPE
    assert g(L, fmt=8, K=40) == ESHAPE    # block size 8 likewise
    assert g(L, fmt=10) == EINVAL
    assert g(L, fmt=-1) == EINVAL


def qd(L, fmt=0, x=P16, rows=32, cols=64, ld=64, rf=0, cf=0, signs=0, rc=P16, rs=P16, rts=P16,
       cc=P16, cs=P16, cts=P16, ws=P16, wsb=4096):
    return L.ifx_quantize_dual(fmt, x, rows, cols, ld, rf, cf, signs, 0, 0, rc, rs, rts, cc, cs, cts,
                               ws, wsb, None)


def test_dual_quantize_validation(L):
    assert qd(L, rf=16) == EINVAL              # the strided bit is implied, not a flag
    assert qd(L, cf=16) == EINVAL
    assert qd(L, cf=1 << 7) == EINVAL
    assert qd(L, signs=1 << 16) == EINVAL
    assert qd(L, fmt=10) == EINVAL
    assert qd(L, rts=None) == EINVAL
    assert qd(L, cts=None) == EINVAL
    assert qd(L, fmt=2) == EUNSUPPORTED        # IF3 / IF6: not training formats
    assert qd(L, fmt=3) == EUNSUPPORTED
    assert qd(L, fmt=7) == EUNSUPPORTED        # block size 8
    assert qd(L, rows=40) == ESHAPE            # both axes are grouped
    assert qd(L, cols=40, ld=40) == ESHAPE
    assert qd(L, ld=48) == ESHAPE
    assert qd(L, rows=-16) == ESHAPE
    assert qd(L, cc=None) == EINVAL
    assert qd(L, rc=P16 + 8) == EALIGN
    assert qd(L, cc=P16 + 8) == EALIGN
    assert qd(L, x=P_ODD) == EALIGN
    assert qd(L, ws=None) == EWORKSPACE
    assert qd(L, wsb=16) == EWORKSPACE
    assert qd(L, ws=P16 + 4) == EALIGN


def test_dequantize_validation(L):
    d = lambda **k: L.if4_dequantize(k.get("codes", P16), P16, k.get("ts", P16),
                                     k.get("rows", 8), k.get("cols", 64), k.get("out", P16),
                                     k.get("dtype", 0), None)
    assert d(cols=40) == ESHAPE
    assert d(out=None) == EINVAL
    assert d(dtype=3) == EINVAL
    assert d(codes=P16 + 2) == EALIGN
    assert d(rows=0) == 0     # empty: nothing to do


def test_empty_gemm_is_noop(L):
    assert g(L, M=0) == 0
    assert g(L, N=0) == 0


def test_oracle_not_linked(L):
    """The product library must not depend on the oracle."""
    import subprocess
    from paper_2603_28765_amd import ops
    out = subprocess.run(["ldd", ops.LIB_PATH], capture_output=True, text=True).stdout
    assert "oracle" not in out
    syms = subprocess.run(["nm", "-D", ops.LIB_PATH], capture_output=True, text=True).stdout
    assert "oracle_" not in syms
