"""Code generation checks on the gfx950 assembly of libmq (no GPU needed).

MFMA results must only be read inside the basic block of the MFMA that wrote
them: the compiler places the wait states a VALU read of an MFMA result needs
reliably within a block, but a read in a successor block right after a
branch has been observed to miss them (stale accumulator values).  The kernels
are written so that every group's MFMA results are converted in the block
that produced them; this test keeps it that way.
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
        cmd = [os.environ.get("HIPCC", "/opt/rocm/bin/hipcc"), *[f for f in build.FLAGS if f not in ("-shared", "-fPIC")],
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


def mfma_escapes(lines):
    """(line index, registers) of MFMA results not consumed in their block."""
    bad = []
    insts = []
    for ln in lines:
        s = ln.strip()
        if not s or s.startswith(";") or s.startswith("."):
            if re.match(r"^\.LBB\S*:", s):
                insts.append(("LABEL", []))
            continue
        insts.append(split_operands(s))
    for i, (op, ops) in enumerate(insts):
        if not op.startswith("v_mfma"):
            continue
        pending = regs(ops[0])
        for op2, ops2 in insts[i + 1:]:
            if op2 == "LABEL" or op2.startswith(_BRANCH):
                break
            if op2.startswith(_ALL_READ):
                pending -= regs(",".join(ops2))
                continue
            srcs = regs(",".join(ops2[1:])) if ops2 else set()
            dst = regs(ops2[0]) if ops2 else set()
            pending -= srcs
            pending -= dst
            if not pending:
                break
        if pending:
            bad.append((i, sorted(pending)))
    return bad


@pytest.fixture(scope="module")
def asm():
    return kernels_asm()


def test_gemm_kernels_have_mfma(asm):
    names = [k for k in asm if "gemm" in k]
    assert any("tiled" in k for k in names) and any("stream" in k for k in names)
    for k in names:
        assert any("v_mfma_f32_16x16x128_f8f6f4" in l for l in asm[k]), k


def test_mfma_results_consumed_in_block(asm):
    problems = {k: mfma_escapes(v) for k, v in asm.items() if "gemm" in k}
    problems = {k: v for k, v in problems.items() if v}
    assert not problems, f"MFMA results read outside their block: {problems}"


def test_no_packed_fp32_instructions(asm):
    for k, lines in asm.items():
        for l in lines:
            assert not re.search(r"\bv_pk_(add|mul|fma)_f32\b", l), (k, l)

