"""The attention kernels read their K and V operands and block-table entries
from LDS with inline-assembly ds_read instructions and wait for them with
explicit s_waitcnt lgkmcnt instructions that name the destination registers.
The compiler does not know such a read is still in flight: if it copies or
reuses a destination register before the wait (for example to build a pair
from a 32-bit result), the copy holds stale contents or the late data lands
on top of another value. A stale block-table entry becomes a garbage block
index and a load from a garbage address.

This test compiles attention.hip for gfx950 to assembly and checks every
attention kernel: inside a basic block, no instruction after an inline-asm
LDS read touches its destination registers before an lgkmcnt wait that
covers the read (CPU only: hipcc cross-compiles)."""
import os
import re
import shutil
import subprocess

import pytest

from paper_2607_03333_amd import build

ROCM = os.environ.get("ROCM_PATH", "/opt/rocm")
HIPCC = os.path.join(ROCM, "bin", "hipcc")


def _vregs(text):
    out = set()
    for m in re.finditer(r"\bv\[(\d+):(\d+)\]|\bv(\d+)\b", text):
        if m.group(3) is not None:
            out.add(int(m.group(3)))
        else:
            out.update(range(int(m.group(1)), int(m.group(2)) + 1))
    return out


def lds_wait_hazards(asm, kernel_pattern=r"attn_bf16"):
    """(kernel, line, instruction) of every use of a pending inline-asm LDS
    read's destination inside its basic block. LDS operations complete in
    order, so lgkmcnt(k) retires all but the k most recent."""
    issues = []
    in_kernel, name, pending, in_asm = False, None, [], False
    for ln, line in enumerate(asm.splitlines(), 1):
        t = line.strip()
        if re.match(r"^_Z\S+:", t):
            name = t.split(":")[0]
            in_kernel, pending = re.search(kernel_pattern, name) is not None, []
            continue
        if not in_kernel:
            continue
        if t.startswith(";;#ASMSTART"):
            in_asm = True
            continue
        if t.startswith(";;#ASMEND"):
            in_asm = False
            continue
        if re.match(r"^(\.LBB\S+:|; %bb\.\d+:)", t):
            pending = []  # a new basic block: this check stays inside one
            continue
        if not t or t.startswith(";") or t.startswith("."):
            continue
        op = t.split()[0]
        args = t.split(None, 1)[1] if " " in t else ""
        if op == "s_waitcnt":
            m = re.search(r"lgkmcnt\((\d+)\)", t)
            if m:
                k = int(m.group(1))
                pending = pending[len(pending) - k:] if 0 < k < len(pending) else ([] if k == 0 else pending)
            continue
        touched = _vregs(args.split(",")[0]) if (op.startswith("ds_read") and in_asm) else _vregs(args)
        if any(regs & touched for regs in pending):
            issues.append((name, ln, t))
        if op.startswith("ds_"):
            pending.append(_vregs(args.split(",")[0]) if (op.startswith("ds_read") and in_asm) else set())
    return issues


def test_scanner_flags_a_copy_of_a_pending_read():
    """The pattern that once built a table-entry pair from a 32-bit read:
    the copy runs before the read has written v5."""
    bad = """_ZN5spork4demoE:
;;#ASMSTART
	ds_read_b32 v5, v2
;;#ASMEND
	v_mov_b32_e32 v4, v5
	s_waitcnt lgkmcnt(0)
	v_readfirstlane_b32 s26, v4
"""
    good = bad.replace("\tv_mov_b32_e32 v4, v5\n\ts_waitcnt lgkmcnt(0)\n", "\ts_waitcnt lgkmcnt(0)\n\tv_mov_b32_e32 v4, v5\n")
    assert lds_wait_hazards(bad, r"demo") == [("_ZN5spork4demoE", 5, "v_mov_b32_e32 v4, v5")]
    assert lds_wait_hazards(good, r"demo") == []


@pytest.mark.skipif(shutil.which(HIPCC) is None and not os.path.exists(HIPCC), reason="hipcc not installed")
def test_attention_kernels_wait_before_using_lds_reads(tmp_path):
    out = tmp_path / "attention.s"
    cmd = [HIPCC, *build.DEVICE_FLAGS, f"-I{build.INCLUDE}", f"-I{build.CSRC}", "--cuda-device-only", "-S",
           "-o", str(out), os.path.join(build.CSRC, "attention.hip")]
    subprocess.run(cmd, check=True, capture_output=True, timeout=600)
    asm = out.read_text()
    assert re.search(r"attn_bf16", asm)
    assert lds_wait_hazards(asm) == []
