"""Register hazards of the asm-managed loads in the fast GEMM kernels.

The fast path issues its A-operand loads and LDS copies as inline asm and
waits for them with explicit `s_waitcnt vmcnt(N)`.  The compiler does not see
those loads as loads, so it never delays a write to, or a read of, a register
that such a load is still filling; the kernel source has to keep every such
register live and untouched until a wait that covers the load.  This test
compiles gemm.hip for gfx950 (device code only, the library's own flags),
replays the vmcnt queue along prologue, two loop iterations and epilogue of
every fast kernel, and fails on any instruction that touches a register of a
load that may still be outstanding.  (A write there once let the last,
unused A prefetch overwrite the epilogue's store address.)
"""
import os
import re
import shutil
import subprocess

import pytest

from paper_2603_28765_amd import _build

HERE = os.path.dirname(os.path.abspath(__file__))


def _regs(text):
    out = set()
    for m in re.finditer(r"\bv\[(\d+):(\d+)\]|\bv(\d+)\b", text):
        if m.group(3):
            out.add(int(m.group(3)))
        else:
            out.update(range(int(m.group(1)), int(m.group(2)) + 1))
    return out


def vmem_violations(lines, loop_header, back_edge):
    """Walk prologue, the loop body twice and the epilogue; return the
    (index, text) of instructions that touch an outstanding load's VGPRs."""
    path = (list(range(0, back_edge + 1)) + list(range(loop_header, back_edge + 1)) * 2
            + list(range(back_edge + 1, len(lines))))
    queue, bad = [], []
    for i in path:
        ln = lines[i].strip()
        if not ln or ln.startswith((".", ";")) or ln.endswith(":"):
            continue
        op = ln.split()[0]
        m = re.match(r"s_waitcnt.*vmcnt\((\d+)\)", ln)
        if m:
            del queue[: max(0, len(queue) - int(m.group(1)))]
            continue
        args = ln.split(None, 1)[1] if " " in ln else ""
        pending = set().union(*queue) if queue else set()
        if not op.startswith("s_") and _regs(args) & pending:
            bad.append((i, ln))
        if op.startswith(("global_load", "buffer_load")):
            queue.append(set() if "lds" in op else _regs(args.split(",")[0]))
        elif op.startswith(("global_store", "buffer_store", "global_atomic")):
            queue.append(set())
    return bad


def test_checker_finds_the_pattern():
    """The replay flags a write into a pending load's registers and accepts
    the same write after a covering wait."""
    asm = ["\tglobal_load_dwordx4 v[10:13], v[40:41], off",
           ".LBB0_1:  ; Inner Loop Header",
           "\tv_add_u32_e32 v1, v2, v3",
           "\ts_cbranch_scc1 .LBB0_1",
           "\tv_mad_u64_u32 v[10:11], s[2:3], v0, s0, 0",
           "\ts_waitcnt vmcnt(0)",
           "\tglobal_store_dword v[10:11], v8, off"]
    assert len(vmem_violations(asm, 1, 3)) == 1
    fixed = asm[:4] + ["\ts_waitcnt vmcnt(0)"] + asm[4:]
    assert vmem_violations(fixed, 1, 3) == []


@pytest.fixture(scope="module")
def gemm_asm(tmp_path_factory):
    hipcc = _build.hipcc()
    if not (shutil.which(hipcc) or os.path.exists(hipcc)):
        pytest.skip("hipcc not available")
    out = str(tmp_path_factory.mktemp("asm") / "gemm.s")
    flags = [f for f in _build.compile_flags() if f != "-fPIC"]
    src = os.path.join(os.path.dirname(_build.__file__), "csrc", "gemm.hip")
    r = subprocess.run([hipcc, *flags, "--cuda-device-only", "-S", src, "-o", out],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    with open(out) as f:
        return f.read()


def test_fast_gemm_kernels_have_no_pending_load_hazards(gemm_asm):
    names = re.findall(r"^(_ZN3ifq12gemm_tn_fast\S+):", gemm_asm, re.M)
    assert len(names) >= 6  # IF4, NVFP4, NVINT4 x {fp32, bf16} out
    for name in names:
        start = gemm_asm.index(name + ":")
        body = gemm_asm[start: gemm_asm.index(".Lfunc_end", start)].split("\n")
        header = next(i for i, ln in enumerate(body) if "Inner Loop Header" in ln)
        back = max(i for i, ln in enumerate(body)
                   if ln.strip().startswith("s_cbranch_scc1") and i > header)
        loads = sum(1 for ln in body if "global_load_dwordx4 v[" in ln)
        assert loads >= 16, (name, loads)
        bad = vmem_violations(body, header, back)
        assert bad == [], (name, bad[:3])
