"""The fused contraction issues its LDS fragment reads, and the global loads of
its U fragments, from inline assembly and waits for them with separate
inline-assembly waits, so the compiler's own wait insertion cannot see them.
Correctness then rests on one property of the generated code: no vector
instruction reads or writes a register that an in-flight ``ds_read_b128`` or
buffer load is still filling.  A register copy placed before the wait (which
the compiler makes, for instance, when one variable is bound to two operands
of the wait) breaks it, and shows up on the GPU only as rare wrong values.

This test compiles the kernel to gfx950 assembly on the CPU, one build per
storage dtype, and checks the property with a forward dataflow pass over the
basic blocks of each kernel.  LDS reads of a wave complete in issue order, so
after ``s_waitcnt lgkmcnt(n)`` only the last n reads issued may still be
pending (scalar loads counted by the same counter only make fewer pending);
likewise vector-memory operations (loads, stores and buffer-to-LDS loads)
under ``vmcnt``.
"""
import os
import re
import subprocess
from concurrent.futures import ThreadPoolExecutor

import pytest

from paper_1905_05233_amd import build_native as B


def _device_asm(source, dtype_code, out_dir):
    out = os.path.join(out_dir, f"{source}_{dtype_code}.s")
    cmd = ([B.HIPCC] + B.COMMON + B.DEVICE + [f"-DWG_DTYPE={dtype_code}", "--cuda-device-only", "-S",
                                                os.path.join(B.CSRC, f"{source}.hip"), "-o", out])
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    with open(out) as f:
        return f.read()


def _vregs(operands):
    regs = set()
    for a, b in re.findall(r"\bv\[(\d+):(\d+)\]", operands):
        regs |= set(range(int(a), int(b) + 1))
    for a in re.findall(r"\bv(\d+)\b", operands):
        regs.add(int(a))
    return regs


def _blocks(code):
    """Basic blocks as (label, instructions); a block ends at a label or a branch."""
    blocks, cur, label = [], [], "entry"
    for line in code.split("\n"):
        s = line.strip()
        m = re.match(r"^(\.LBB\w+):", s)
        if m:
            blocks.append((label, cur))
            label, cur = m.group(1), []
            continue
        if not s or s.startswith(";"):
            continue
        ins = s.split(";")[0].strip()
        if not ins:
            continue
        cur.append(ins)
        if ins.startswith(("s_cbranch", "s_branch")):
            blocks.append((label, cur))
            label, cur = f"after{len(blocks)}", []
    blocks.append((label, cur))
    return blocks


def _vmem_dest(ins):
    """Destination registers of a vector-memory load into VGPRs (none for stores
    and for the buffer-to-LDS form, whose first operand is an address)."""
    m = re.match(r"^(buffer|global|flat)_load_\w+\s+(v\[(\d+):(\d+)\]|v(\d+))", ins)
    if not m or ins.rstrip().endswith(" lds"):
        return frozenset()
    if m.group(3) is not None:
        return frozenset(range(int(m.group(3)), int(m.group(4)) + 1))
    return frozenset([int(m.group(5))])


def lds_read_hazards(asm):
    """(kernel, instruction) pairs that touch a register of an LDS read or a
    vector-memory load in flight."""
    body = asm[:asm.index("amdhsa.kernels")] if "amdhsa.kernels" in asm else asm
    parts = re.split(r"\n(_Z\S+):[^\n]*\n", body)
    found, kernels = [], 0
    for i in range(1, len(parts), 2):
        name, code = parts[i], parts[i + 1]
        kernels += 1
        blocks = _blocks(code)
        index = {label: k for k, (label, _) in enumerate(blocks)}
        succ = []
        for k, (_, ins) in enumerate(blocks):
            nxt = []
            last = ins[-1] if ins else ""
            m = re.match(r"^s_c?branch\w*\s+(\.LBB\w+)", last)
            if m:
                nxt.append(index[m.group(1)])
            if not last.startswith(("s_branch", "s_endpgm", "s_setpc")) and k + 1 < len(blocks):
                nxt.append(k + 1)
            succ.append(nxt)
        # state: for each depth d (0 = youngest), the registers of reads that may
        # be pending with d younger reads issued after them; merged by union
        # two in-order queues (LDS reads under lgkmcnt, vector memory under vmcnt)
        depth = 64
        empty = tuple(frozenset() for _ in range(depth))
        entry = [(empty, empty) for _ in blocks]
        work, hits = list(range(len(blocks))), set()
        while work:
            k = work.pop(0)
            lgkm, vm = list(entry[k][0]), list(entry[k][1])
            for ins in blocks[k][1]:
                live = frozenset().union(*lgkm, *vm)
                if live and not ins.startswith("s_"):
                    operands = ins.split(None, 1)[1] if " " in ins else ""
                    regs = _vregs(operands)
                    if ins.startswith(("buffer_", "global_", "flat_")):
                        regs = regs - _vmem_dest(ins)   # a load's own destination is not a use
                    if regs & live:
                        hits.add((name, ins))
                m = re.match(r"^ds_read_b128\s+v\[(\d+):(\d+)\]", ins)
                if m:
                    lgkm = [frozenset(range(int(m.group(1)), int(m.group(2)) + 1))] + lgkm[:depth - 1]
                    continue
                if ins.startswith(("buffer_", "global_", "flat_")):
                    vm = [_vmem_dest(ins)] + vm[:depth - 1]
                    continue
                if ins.startswith("s_waitcnt"):
                    w = re.search(r"lgkmcnt\((\d+)\)", ins)
                    if w:
                        n = int(w.group(1))
                        lgkm = lgkm[:n] + [frozenset()] * (depth - n)
                    w = re.search(r"vmcnt\((\d+)\)", ins)
                    if w:
                        n = int(w.group(1))
                        vm = vm[:n] + [frozenset()] * (depth - n)
            for j in succ[k]:
                new = (tuple(a | b for a, b in zip(entry[j][0], lgkm)), tuple(a | b for a, b in zip(entry[j][1], vm)))
                if new != entry[j]:
                    entry[j] = new
                    if j not in work:
                        work.append(j)
        found.extend(sorted(hits))
    return kernels, found


def test_scanner_flags_a_copy_before_the_wait():
    """The scanner itself: a copy of an in-flight fragment across a branch is found,
    the same code with the wait first is not; a counted wait covers all but the
    youngest reads."""
    bad = """
_Zk:                                    ; @_Zk
\tds_read_b128 v[12:15], v48
\ts_cbranch_vccnz .LBB0_2
\tv_add_f32_e32 v7, v11, v7
.LBB0_2:
\tv_mov_b64_e32 v[8:9], v[12:13]
\ts_waitcnt lgkmcnt(0)
\tv_mfma_f32_16x16x32_bf16 v[0:3], v[8:11], v[12:15], 0
\ts_endpgm
"""
    good = bad.replace("\tv_mov_b64_e32 v[8:9], v[12:13]\n\ts_waitcnt lgkmcnt(0)\n",
                       "\ts_waitcnt lgkmcnt(0)\n\tv_mov_b64_e32 v[8:9], v[12:13]\n")
    assert lds_read_hazards(bad) == (1, [("_Zk", "v_mov_b64_e32 v[8:9], v[12:13]")])
    assert lds_read_hazards(good) == (1, [])
    counted = """
_Zk:                                    ; @_Zk
\tds_read_b128 v[12:15], v48
\tds_read_b128 v[16:19], v49
\tds_read_b128 v[20:23], v50
\ts_waitcnt lgkmcnt(1)
\tv_mfma_f32_16x16x32_bf16 v[0:3], v[12:15], v[16:19], 0
\tv_mov_b32_e32 v24, v21
\ts_endpgm
"""
    assert lds_read_hazards(counted) == (1, [("_Zk", "v_mov_b32_e32 v24, v21")])
    vmem = """
_Zk:                                    ; @_Zk
\tbuffer_load_dwordx4 v[12:15], v40, s[0:3], 0 offen
\tbuffer_load_dwordx4 v1, s[4:7], 0 offen lds
\tbuffer_load_dwordx4 v[16:19], v41, s[0:3], 0 offen
\ts_waitcnt vmcnt(2)
\tv_mov_b32_e32 v20, v13
\tv_mov_b32_e32 v21, v17
\ts_endpgm
"""
    assert lds_read_hazards(vmem) == (1, [("_Zk", "v_mov_b32_e32 v21, v17")])


@pytest.fixture(scope="module")
def fused_asm(tmp_path_factory):
    """gfx950 assembly of fused.hip, one build per storage dtype (the source is
    compiled with WG_DTYPE set)."""
    if not os.path.exists(B.HIPCC):
        pytest.skip("hipcc not installed")
    out = str(tmp_path_factory.mktemp("fused_asm"))
    with ThreadPoolExecutor(3) as ex:
        return dict(zip((0, 1, 2), ex.map(lambda d: _device_asm("fused", d, out), (0, 1, 2))))


def test_kernels_wait_before_using_lds_fragments(fused_asm):
    for code, asm in fused_asm.items():
        kernels, hits = lds_read_hazards(asm)
        assert kernels >= 40, f"fused dtype {code}: only {kernels} kernels found in the assembly"
        assert not hits, f"fused dtype {code}: {len(hits)} uses of in-flight LDS fragments, e.g. {hits[:3]}"


def stage_wait_violations(kernel_code, per_step, steps):
    """For a kernel whose first ``steps`` workgroup barriers each begin a step,
    and whose buffer-to-LDS loads fill the stages in step order, ``per_step``
    loads per wave and step: the steps at which the last vmcnt wait before the
    barrier does not cover that step's loads, as (step, vector-memory
    operations issued after the step's last load, wait)."""
    vm, nbar, wait, bad = [], 0, None, []
    for line in kernel_code.split("\n"):
        s = line.strip()
        if not s or s.startswith((";", ".")):
            continue
        ins = s.split(";")[0].strip()
        if ins.startswith(("buffer_load", "global_load")):
            vm.append(ins.endswith(" lds"))
        m = re.match(r"s_waitcnt.*vmcnt\((\d+)\)", ins)
        if m:
            wait = int(m.group(1))
        if ins.startswith("s_barrier") and nbar < steps:
            lds = [i for i, is_lds in enumerate(vm) if is_lds]
            last = (nbar + 1) * per_step - 1
            after = len(vm) - 1 - lds[last] if last < len(lds) else -1
            if wait is None or after < wait:
                bad.append((nbar, after, wait))
            nbar += 1
            wait = None
    return nbar, bad


def test_scanner_counts_stage_waits():
    """The stage-wait scanner on hand-written code: the load of step 1 needs
    two younger loads when the wait allows two outstanding."""
    ok = """
\tbuffer_load_dwordx4 v1, s[4:7], 0 offen lds
\tbuffer_load_dwordx4 v1, s[8:11], 0 offen lds
\tbuffer_load_dwordx4 v[2:5], v6, s[0:3], 0 offen
\ts_waitcnt vmcnt(2)
\ts_barrier
\tbuffer_load_dwordx4 v[8:11], v6, s[0:3], 0 offen
\ts_waitcnt vmcnt(2)
\ts_barrier
"""
    assert stage_wait_violations(ok, 1, 2) == (2, [])
    assert stage_wait_violations(ok.replace("vmcnt(2)\n\ts_barrier\n\tbuffer_load_dwordx4 v[8:11]",
                                            "vmcnt(3)\n\ts_barrier\n\tbuffer_load_dwordx4 v[8:11]"), 1, 2) == (2, [(0, 2, 3)])
    # two loads per step: the wait before the first barrier must cover both
    assert stage_wait_violations(ok, 2, 1) == (1, [(0, 1, 2)])


def test_scanner_checks_looped_stage_waits():
    """The looped form's checker on a hand-written loop: one group of two
    loads per step after a prologue of two groups (three stages); a wait that
    leaves two groups outstanding, or a path that issues two groups between
    barriers, is flagged."""
    code = """
_Zk:                                    ; @_Zk
\tbuffer_load_dwordx4 v1, s[4:7], 0 offen lds
\tbuffer_load_dwordx4 v1, s[4:7], 0 offen lds
\tbuffer_load_dwordx4 v1, s[4:7], 0 offen lds
\tbuffer_load_dwordx4 v1, s[4:7], 0 offen lds
.LBB0_1:
\ts_waitcnt vmcnt(2)
\ts_barrier
\tbuffer_load_dwordx4 v1, s[4:7], 0 offen lds
\tbuffer_load_dwordx4 v1, s[4:7], 0 offen lds
\ts_cbranch_scc1 .LBB0_1
\ts_waitcnt vmcnt(0)
\ts_barrier
\ts_endpgm
"""
    assert chunked_wait_violations(code, 2, 3) == []
    assert chunked_wait_violations(code.replace("vmcnt(2)", "vmcnt(4)"), 2, 3)
    extra = code.replace("\ts_cbranch_scc1 .LBB0_1", "\ts_cbranch_scc1 .LBB0_1\n\tbuffer_load_dwordx4 v1, s[4:7], 0 offen lds\n"
                         "\tbuffer_load_dwordx4 v1, s[4:7], 0 offen lds\n\ts_branch .LBB0_1")
    assert chunked_wait_violations(extra, 2, 3)


def test_unrolled_kernels_wait_for_their_stage(fused_asm):
    """The unrolled kernels count their own vmcnt waits: before step s's
    barrier, this wave's buffer-to-LDS loads of step s (3 per 128-byte slice,
    the s-th group in issue order) must have completed, i.e. at least as many
    vector-memory operations were issued after the group's last load as the
    wait leaves outstanding.  The template arguments give alpha', the
    slices per step, the domain points per step and the steps per domain
    point (steps = alpha'^2 / the points per step, rounded up, times the
    steps per point)."""
    for code, asm in fused_asm.items():
        body = asm[:asm.index("amdhsa.kernels")] if "amdhsa.kernels" in asm else asm
        parts = re.split(r"\n(_Z\S+):[^\n]*\n", body)
        seen = 0
        for i in range(1, len(parts), 2):
            m = re.search(r"contract_output_unrolled_kernelILi\d+ELi\d+ELi(\d+)E.*ELi(\d)ELi(\d)ELb([01])ELi(\d)EEEv",
                          parts[i])
            if not m:
                continue
            seen += 1
            alpha, nsl, xp, ch = int(m.group(1)), int(m.group(2)), int(m.group(3)), m.group(4) == "1"
            nck = int(m.group(5))
            if ch:
                bad = chunked_wait_violations(parts[i + 1], 3 * nsl, 4 if nsl == 1 else 3)
                assert not bad, f"dtype {code}: {parts[i][:80]}: {bad[:3]}"
                continue
            n = -(-alpha * alpha // xp) * nck
            steps, bad = stage_wait_violations(parts[i + 1], 3 * nsl, n)
            assert steps == n, f"dtype {code}: {parts[i][:80]}: {steps} step barriers"
            assert not bad, f"dtype {code}: {parts[i][:80]}: stage loads not covered {bad[:3]}"
        assert seen >= 59, f"dtype {code}: {seen} unrolled kernels"


def chunked_wait_violations(kernel_code, per_step, stages):
    """The unrolled kernel's long-row form runs its steps in loops, one group
    of ``per_step`` buffer-to-LDS loads per step after ``stages - 1`` groups in
    the prologue, and waits for the same count before every step's barrier.
    On every path through the kernel's control-flow graph that requires: the
    first barrier follows the prologue's groups, every later step barrier
    follows exactly one group, and every step's wait leaves at most
    ``stages - 2`` groups outstanding (so the step's own group, ``stages - 1``
    behind the newest, has landed).  The steps end at the wait for every load
    (vmcnt(0)) before the epilogue.  Returns the violations found."""
    blocks = _blocks(kernel_code)
    index = {label: k for k, (label, _) in enumerate(blocks)}
    succ = []
    for k, (_, ins) in enumerate(blocks):
        nxt = []
        last = ins[-1] if ins else ""
        m = re.match(r"^s_c?branch\w*\s+(\.LBB\w+)", last)
        if m:
            nxt.append(index[m.group(1)])
        if not last.startswith(("s_branch", "s_endpgm", "s_setpc")) and k + 1 < len(blocks):
            nxt.append(k + 1)
        succ.append(nxt)
    # state: (barriers seen, loads since the last barrier, last vmcnt since it); "done" after the final wait
    entry = [set() for _ in blocks]
    entry[0].add((False, 0, None))
    work, bad, steps = [0], [], 0
    while work:
        k = work.pop()
        for st in list(entry[k]):
            cur = st
            for ins in blocks[k][1]:
                if cur == "done":
                    break
                seen, loads, wait = cur
                if ins.startswith(("buffer_load", "global_load")) and ins.endswith(" lds"):
                    cur = (seen, loads + 1, wait)
                    continue
                m = re.match(r"s_waitcnt.*vmcnt\((\d+)\)", ins)
                if m:
                    n = int(m.group(1))
                    cur = "done" if (n == 0 and seen) else (seen, loads, n)
                    continue
                if ins.startswith("s_barrier"):
                    want = per_step * (stages - 1) if not seen else per_step
                    if loads != want:
                        bad.append(("loads before barrier", blocks[k][0], loads, want))
                    if wait is None or wait > per_step * (stages - 2):
                        bad.append(("wait", blocks[k][0], wait))
                    steps += 1
                    cur = (True, 0, None)
            for j in succ[k]:
                if cur not in entry[j]:
                    entry[j].add(cur)
                    work.append(j)
        if len(bad) > 20:
            break
    if steps < 2:
        bad.append(("steps", steps))
    return bad
