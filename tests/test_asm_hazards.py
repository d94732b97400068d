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


def _loop_bounds(body):
    """(header, back edge) of the K loop: the line of the label marked
    "Inner Loop Header" and the last conditional branch back to it."""
    header = next(i for i, ln in enumerate(body) if "Inner Loop Header" in ln)
    label = body[header].split(":")[0].strip()
    back = max(i for i, ln in enumerate(body)
               if ln.strip().startswith("s_cbranch_") and ln.split()[-1] == label and i > header)
    return header, back


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
    assert len(names) >= 12  # IF4, NVFP4, NVINT4, IF3, IF4-BS8, NVFP4-BS8 x {fp32, bf16} out
    for name in names:
        start = gemm_asm.index(name + ":")
        body = gemm_asm[start: gemm_asm.index(".Lfunc_end", start)].split("\n")
        header, back = _loop_bounds(body)
        loads = sum(1 for ln in body if "global_load_dwordx4 v[" in ln or "global_load_dwordx2 v[" in ln)
        assert loads >= 16, (name, loads)
        bad = vmem_violations(body, header, back)
        assert bad == [], (name, bad[:3])


# ----------------------------------------------------------------- LDS side
# The copies into LDS (global_load_lds_dwordx4) are asm too.  Their data is
# safe to read once the copying wave has drained them with a vmcnt wait and
# every wave has passed a barrier after that, and a slot may be refilled only
# after a barrier that follows its last read.  Two checks: the compiled code
# drains every copy before the second barrier after its issue (so it is
# visible one barrier period later), and the slot schedule of the kernel
# reads every chunk at least one barrier after that and refills a slot only
# after its last read.

def lds_copy_violations(lines, loop_header, back_edge):
    """At every s_barrier along prologue, two loop iterations and epilogue,
    return the copies into LDS still outstanding that were issued before the
    previous barrier."""
    path = (list(range(0, back_edge + 1)) + list(range(loop_header, back_edge + 1)) * 2
            + list(range(back_edge + 1, len(lines))))
    queue, bad, barriers = [], [], 0
    for i in path:
        ln = lines[i].strip()
        if not ln or ln.startswith((".", ";")) or ln.endswith(":"):
            continue
        op = ln.split()[0]
        m = re.match(r"s_waitcnt.*vmcnt\((\d+)\)", ln)
        if m:
            del queue[: max(0, len(queue) - int(m.group(1)))]
            continue
        if op == "s_barrier":
            bad += [(i, q) for q in queue if q is not None and q < barriers]
            barriers += 1
        elif op.startswith(("global_load", "buffer_load")):
            queue.append(barriers if "lds" in op else None)
        elif op.startswith(("global_store", "buffer_store", "global_atomic")):
            queue.append(None)
    return bad


def test_lds_checker_finds_the_pattern():
    asm = ["\tglobal_load_lds_dwordx4 v[6:7], off",
           "\ts_barrier",
           ".LBB0_1:  ; Inner Loop Header",
           "\tv_add_u32_e32 v1, v2, v3",
           "\ts_cbranch_scc1 .LBB0_1",
           "\ts_barrier"]
    assert len(lds_copy_violations(asm, 2, 4)) == 1
    fixed = asm[:5] + ["\ts_waitcnt vmcnt(0)"] + asm[5:]
    assert lds_copy_violations(fixed, 2, 4) == []


def test_fast_gemm_copies_are_drained_within_one_barrier_period(gemm_asm):
    names = re.findall(r"^(_ZN3ifq12gemm_tn_fast\S+):", gemm_asm, re.M)
    assert len(names) >= 6
    for name in names:
        start = gemm_asm.index(name + ":")
        body = gemm_asm[start: gemm_asm.index(".Lfunc_end", start)].split("\n")
        header, back = _loop_bounds(body)
        assert sum(1 for ln in body if "global_load_lds_dwordx4" in ln) >= 6, name
        assert sum(1 for ln in body if ln.strip() == "s_barrier") >= 4, name
        bad = lds_copy_violations(body, header, back)
        assert bad == [], (name, bad[:3])


def _fast_gemm_lds_events(nch, spg=1):
    """The copy and read schedule of the fast GEMM's raw-code and scale slots
    for K = 128 nch (nch % 4 == 0), as the kernel issues it (spg: scale bytes
    per 16 values; block size 8 has 2 and 4-step scale chunks): a list of
    (phase, kind, region, data) with phase the number of barriers passed
    before the event, kind 'copy' or 'read', region (slot kind, slot, half)
    and data the chunk it holds or needs (None: past the end, never used).
    Even steps end with a vmcnt wait that drains every copy issued before
    them: a copy issued in phase p (step p - 2) is drained before the barrier
    that ends the first even step from then on, and the prologue's before
    the first barrier."""
    cps = 4 if spg == 1 else 2          # code chunks per scale chunk
    nsc = nch // cps
    ev = []
    # prologue: B chunks 0, 1; scale chunk 0 (A and B halves), scale chunk 1's
    # A half (block size 8: its B half too)
    ev += [(0, "copy", ("raw", 0, 0), 0), (0, "copy", ("raw", 1, 0), min(1, nch - 1)),
           (0, "copy", ("scl", 0, 0), 0), (0, "copy", ("scl", 0, 1), 0),
           (0, "copy", ("scl", 1, 0), min(1, nsc - 1))]
    if spg == 2:
        ev.append((0, "copy", ("scl", 1, 1), min(1, nsc - 1)))
    # (vmcnt(0); barrier 1) reads of B steps 0, 1, 2 and the A scales of chunk 0
    def read_b(phase, sd):
        c = sd >> 1
        ok = c < nch
        e = c // cps
        return [(phase, "read", ("raw", c & 1, 0), c if ok else None),
                (phase, "read", ("scl", e & 1, 1), e if ok else None)]
    for sd in (0, 1, 2):
        ev += read_b(1, sd)
    ev.append((1, "read", ("scl", 0, 0), 0))
    # (barrier 2) the odd step before step 0: B chunk 2 into raw slot 0
    ev.append((2, "copy", ("raw", 0, 0), min(2, nch - 1)))
    for s in range(2 * nch):
        phase = 2 + s            # barriers passed before step s
        q, c = s % 4, s >> 1
        j, cs = q & 1, q >> 1
        if j == 1:
            ev.append((phase, "copy", ("raw", cs ^ 1, 0), min(c + 3, nch - 1)))
            if spg == 1 and q == 1:
                u = s >> 2
                e = (u + 3) >> 1
                ev.append((phase, "copy", ("scl", e & 1, (u + 1) & 1), min(e, nsc - 1)))
            elif spg == 2:
                e = (s >> 2) + 2
                ev.append((phase, "copy", ("scl", e & 1, q >> 1), min(e, nsc - 1)))
        else:
            ca = min(c + 1, nch - 1)
            ev.append((phase, "read", ("scl", (ca // cps) & 1, 0), ca // cps))
        ev += read_b(phase, s + 3)
    return ev


def _check_lds_schedule(ev):
    """Every read sees its chunk, copied and drained at least one barrier
    earlier, and no copy of other data into that slot is issued before the
    read's barrier.  (Past the last chunk the kernel clamps its copy indices,
    so a slot can be rewritten with the bytes it already holds; such a copy
    changes nothing a read can see.)"""
    problems = []
    for idx, (ph, kind, reg, data) in enumerate(ev):
        if kind != "read" or data is None:
            continue
        copies = [(p, d) for (p, k, r, d) in ev[:idx] if k == "copy" and r == reg]
        if not copies:
            problems.append(("never copied", ph, reg, data))
            continue
        if copies[-1][1] != data:
            problems.append(("slot holds another chunk", ph, reg, data, copies[-1][1]))
            continue
        # the copy that brought this data in (identical rewrites after it change nothing)
        k = len(copies) - 1
        while k > 0 and copies[k - 1][1] == data:
            k -= 1
        p_last = copies[k][0]
        # first phase in which the copy is drained and fenced
        visible = 1 if p_last == 0 else (p_last + 1 if (p_last - 2) % 2 == 0 else p_last + 2)
        if ph < visible:
            problems.append(("read before the copy is drained and fenced", ph, reg, data, p_last))
        same_phase = [p for (p, k, r, d) in ev[idx + 1:] if k == "copy" and r == reg and p <= ph and d != data]
        if same_phase:
            problems.append(("slot refilled before the read's barrier", ph, reg, data))
    return problems


def test_fast_gemm_lds_slot_schedule():
    for spg in (1, 2):
        for nch in (4, 8, 12, 32):
            assert _check_lds_schedule(_fast_gemm_lds_events(nch, spg)) == [], (spg, nch)


def test_lds_schedule_checker_finds_a_slot_reused_too_early():
    ev = _fast_gemm_lds_events(8)
    # move the first main-loop copy into raw slot 1 one phase earlier
    i = next(i for i, e in enumerate(ev) if e[1] == "copy" and e[2] == ("raw", 1, 0) and e[0] > 2)
    p, k, r, d = ev[i]
    bad = ev[:i] + [(p - 1, k, r, d)] + ev[i + 1:]
    bad.sort(key=lambda e: e[0])
    assert _check_lds_schedule(bad) != []
