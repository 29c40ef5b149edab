"""Code generation checks on the gfx950 assembly of libmq (no GPU needed).

A VALU read (or overwrite) of an MFMA result needs wait states after the MFMA:
8 for the fp6 x fp6 f8f6f4 MFMA, 12 when an operand is fp8 (the counts the
compiler itself inserts before such a read in the MFMA's own block).  A read in
a successor block right after a branch has been observed to miss them once
(stale accumulator values), so this test checks every read of an MFMA result
that is reached across a block boundary (a label or a branch): on every path
of the control-flow graph it must come at least that many wait states after
the MFMA (each instruction is one wait state, s_nop n is n + 1).  Reads inside
the MFMA's own block are left to the compiler.
"""
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

_REG = re.compile(r"\b([va])(\d+)\b|\b([va])\[(\d+):(\d+)\]")
_BRANCH = ("s_branch", "s_cbranch", "s_setpc", "s_endpgm", "s_trap")
_ALL_READ = ("ds_write", "ds_store", "global_store", "buffer_store", "flat_store",
             "ds_add", "global_atomic", "buffer_atomic", "s_")


def regs(text):
    out = set()
    for m in _REG.finditer(text):
        if m.group(1):
            out.add(f"{m.group(1)}{m.group(2)}")
        else:
            for r in range(int(m.group(4)), int(m.group(5)) + 1):
                out.add(f"{m.group(3)}{r}")
    return out


def split_operands(line):
    parts = line.split(None, 1)
    if len(parts) < 2:
        return parts[0], []
    ops = [o.strip() for o in re.split(r",(?![^\[]*\])", parts[1].split(";")[0])]
    return parts[0], ops


def kernels_asm():
    from paper_2606_15652_amd import build
    out = {}
    for src in build.sources():
        cmd = [os.environ.get("HIPCC", "/opt/rocm/bin/hipcc"), *[f for f in build.compile_flags(src) if f != "-fPIC"],
               "--cuda-device-only", "-S", src, "-o", "-"]
        asm = subprocess.run(cmd, capture_output=True, text=True, check=True).stdout
        cur = None
        for line in asm.splitlines():
            m = re.match(r"^(_Z\S+|mq\S*):\s", line + " ")
            if m and not line.startswith("\t"):
                cur = m.group(1)
                out[cur] = []
                continue
            if cur is not None:
                if line.strip().startswith(".Lfunc_end"):
                    cur = None
                    continue
                out[cur].append(line)
    return out


def required_wait_states(ops):
    """Wait states before a VALU touches the result of this f8f6f4 MFMA."""
    mods = " ".join(ops)
    cbsz = re.search(r"cbsz:(\d)", mods)
    blgp = re.search(r"blgp:(\d)", mods)
    fp6_or_fp4 = lambda m: m is not None and int(m.group(1)) >= 2
    return 8 if fp6_or_fp4(cbsz) and fp6_or_fp4(blgp) else 12


def _parse(lines):
    """Instructions as (op, operands); labels as ("LABEL", name)."""
    insts = []
    for ln in lines:
        s = ln.strip()
        if not s or s.startswith(";"):
            continue
        m = re.match(r"^(\.LBB\S*):", s)
        if m:
            insts.append(("LABEL", m.group(1)))
            continue
        if s.startswith("."):
            continue
        insts.append(split_operands(s))
    return insts


def _successors(insts):
    where = {ops: i for i, (op, ops) in enumerate(insts) if op == "LABEL"}
    succ = []
    for i, (op, ops) in enumerate(insts):
        if op == "s_branch":
            succ.append([where[ops[0]]])
        elif op.startswith("s_cbranch"):
            succ.append([i + 1, where[ops[0]]])
        elif op.startswith(("s_endpgm", "s_setpc", "s_trap")):
            succ.append([])
        else:
            succ.append([i + 1] if i + 1 < len(insts) else [])
    return succ


def _touches(op, ops, pending):
    """Registers of `pending` that the instruction reads or writes."""
    if op == "LABEL" or not ops:
        return set()
    if op.startswith(_ALL_READ):
        return pending & regs(",".join(ops))
    return pending & (regs(",".join(ops[1:])) | regs(ops[0]))


def _cost(op, ops):
    if op == "LABEL":
        return 0
    if op == "s_nop":
        return int(ops[0], 0) + 1
    return 1


def mfma_escapes(lines):
    """(instruction index, registers, wait states) of MFMA results first
    touched across a block boundary fewer than the required wait states after
    the MFMA, on some path."""
    import heapq
    insts = _parse(lines)
    succ = _successors(insts)
    bad = []
    for i, (op, ops) in enumerate(insts):
        if not op.startswith("v_mfma"):
            continue
        pending = regs(ops[0])
        need = required_wait_states(ops)
        # straight-line part of the block: the compiler's wait states hold
        j = i + 1
        crossed_at = None
        while j < len(insts):
            op2, ops2 = insts[j]
            if op2 == "LABEL":
                crossed_at = j
                break
            pending -= _touches(op2, ops2, pending)
            if not pending:
                break
            if op2.startswith(_BRANCH):
                crossed_at = j
                break
            j += 1
        if not pending or crossed_at is None:
            continue
        # every path from the block boundary on: shortest distance to the
        # first instruction touching a pending register
        dist0 = sum(_cost(*insts[k]) for k in range(i + 1, crossed_at + 1))
        starts = [crossed_at] if insts[crossed_at][0] == "LABEL" else succ[crossed_at]
        best = {}
        heap = [(dist0 + (0 if insts[crossed_at][0] == "LABEL" else 0), k) for k in starts]
        heapq.heapify(heap)
        while heap:
            d, k = heapq.heappop(heap)
            if k in best and best[k] <= d:
                continue
            best[k] = d
            op2, ops2 = insts[k]
            hit = _touches(op2, ops2, pending)
            if hit:
                if d < need:
                    bad.append((i, sorted(hit), d))
                continue
            for n in succ[k]:
                heapq.heappush(heap, (d + _cost(op2, ops2), n))
    return bad


@pytest.fixture(scope="module")
def asm():
    return kernels_asm()


def test_gemm_kernels_have_mfma(asm):
    names = [k for k in asm if "gemm" in k]
    assert any("tiled" in k for k in names) and any("stream" in k for k in names)
    for k in names:
        assert any("v_mfma_f32_16x16x128_f8f6f4" in l for l in asm[k]), k


def test_mfma_results_read_across_blocks_are_far(asm):
    problems = {k: mfma_escapes(v) for k, v in asm.items() if "gemm" in k}
    problems = {k: v for k, v in problems.items() if v}
    assert not problems, f"MFMA results read across a block boundary too soon: {problems}"


def test_escape_check_sees_a_near_read():
    # a read right after a branch join, one wait state after the MFMA on the taken path
    lines = ["v_mfma_f32_16x16x128_f8f6f4 v[0:3], v[4:9], v[10:15], 0 cbsz:2 blgp:2",
             "s_cbranch_scc1 .LBB0_1", "v_mov_b32 v20, 1", ".LBB0_1:",
             "v_add_f32 v21, v0, v1", "s_endpgm"]
    assert [b[1] for b in mfma_escapes(lines)] == [["v0", "v1"]]
    far = lines[:1] + ["s_nop 6"] + lines[1:]     # 8 on the taken path
    assert mfma_escapes(far) == []
    fp8 = [lines[0].replace(" cbsz:2 blgp:2", "")] + far[1:]
    assert [b[1] for b in mfma_escapes(fp8)] == [["v0", "v1"]]


def test_no_packed_fp32_instructions(asm):
    for k, lines in asm.items():
        for l in lines:
            assert not re.search(r"\bv_pk_(add|mul|fma)_f32\b", l), (k, l)

