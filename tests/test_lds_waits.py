"""The fused contraction issues its LDS fragment reads from inline assembly and
waits for them with a separate inline-assembly wait, so the compiler's own
wait insertion cannot see them.  Correctness then rests on one property of
the generated code: no vector instruction reads or writes a register that an
in-flight ``ds_read_b128`` is still filling.  A register copy placed before
the wait (which the compiler makes, for instance, when one variable is bound
to two operands of the wait) breaks it, and shows up on the GPU only as rare
wrong values.

This test compiles the kernel to gfx950 assembly on the CPU, one build per
storage dtype, and checks the property with a forward dataflow pass over the
basic blocks of each kernel (a register is pending from its read until the
next ``s_waitcnt lgkmcnt(0)`` on every path).
"""
import os
import re
import subprocess
from concurrent.futures import ThreadPoolExecutor

import pytest

from paper_1905_05233_amd import build_native as B

FUSED = os.path.join(B.CSRC, "fused.hip")


def _device_asm(dtype_code, out_dir):
    out = os.path.join(out_dir, f"fused_{dtype_code}.s")
    cmd = ([B.HIPCC] + B.COMMON + B.DEVICE + [f"-DWG_DTYPE={dtype_code}", "--cuda-device-only", "-S", FUSED,
                                                "-o", out])
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


def lds_read_hazards(asm):
    """(kernel, instruction) pairs that touch a register of an LDS read in flight."""
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
        entry = [set() for _ in blocks]
        work, hits = list(range(len(blocks))), set()
        while work:
            k = work.pop(0)
            pending = set(entry[k])
            for ins in blocks[k][1]:
                m = re.match(r"^ds_read_b128\s+v\[(\d+):(\d+)\]", ins)
                if m:
                    pending |= set(range(int(m.group(1)), int(m.group(2)) + 1))
                    continue
                if ins.startswith("s_waitcnt") and "lgkmcnt(0)" in ins:
                    pending = set()
                    continue
                if pending and not ins.startswith("s_"):
                    operands = ins.split(None, 1)[1] if " " in ins else ""
                    if _vregs(operands) & pending:
                        hits.add((name, ins))
            for j in succ[k]:
                if not pending <= entry[j]:
                    entry[j] |= pending
                    if j not in work:
                        work.append(j)
        found.extend(sorted(hits))
    return kernels, found


def test_scanner_flags_a_copy_before_the_wait():
    """The scanner itself: a copy of an in-flight fragment across a branch is found,
    the same code with the wait first is not."""
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


@pytest.mark.skipif(not os.path.exists(B.HIPCC), reason="hipcc not installed")
def test_fused_kernel_waits_before_using_lds_fragments(tmp_path):
    with ThreadPoolExecutor(3) as ex:
        asms = list(ex.map(lambda d: _device_asm(d, str(tmp_path)), [0, 1, 2]))
    for code, asm in enumerate(asms):
        kernels, hits = lds_read_hazards(asm)
        assert kernels >= 40, f"dtype {code}: only {kernels} kernels found in the assembly"
        assert not hits, f"dtype {code}: {len(hits)} uses of in-flight LDS fragments, e.g. {hits[:3]}"
