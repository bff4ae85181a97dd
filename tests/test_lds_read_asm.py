"""The tile loops issue some LDS reads as inline assembly (so that the
compiler does not wait for DMA into other stages) and end each batch with an
s_waitcnt lgkmcnt(0) that names the read values as operands.  Until that wait
a read's destination registers are still being written by the LDS, so no
compiler-generated instruction may touch them in between.  This test builds
the gfx950 assembly of the library (host only, no GPU) and checks that."""

import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _regs(operand: str) -> set:
    out = set()
    for m in re.finditer(r"v\[(\d+):(\d+)\]|v(\d+)", operand):
        if m.group(3):
            out.add(int(m.group(3)))
        else:
            out.update(range(int(m.group(1)), int(m.group(2)) + 1))
    return out


def scan(asm_lines):
    """(kernels with inline LDS reads, offending instructions per kernel)."""
    cur, inasm, pend = None, False, set()
    kernels, bad = set(), {}
    for line in asm_lines:
        m = re.match(r"^(_Z\S+):", line)
        if m:
            cur, pend = m.group(1), set()
            continue
        t = line.strip()
        if t.startswith(";;#ASMSTART"):
            inasm = True
            continue
        if t.startswith(";;#ASMEND"):
            inasm = False
            continue
        if not t or t.startswith((";", ".")):
            continue
        if inasm and t.startswith("ds_read"):
            kernels.add(cur)
            pend |= _regs(t.split()[1].rstrip(","))
            continue
        if inasm and t.startswith("s_waitcnt") and "lgkmcnt(0)" in t:
            pend = set()
            continue
        if pend and _regs(t) & pend:
            bad.setdefault(cur, []).append(t)
    return kernels, bad


def test_scan_flags_a_touched_register():
    lines = ["_Zk:", ";;#ASMSTART", "ds_read_b128 v[4:7], v1", ";;#ASMEND",
             "v_mov_b32 v8, v5", ";;#ASMSTART", "s_waitcnt lgkmcnt(0)", ";;#ASMEND"]
    kernels, bad = scan(lines)
    assert kernels == {"_Zk"} and bad == {"_Zk": ["v_mov_b32 v8, v5"]}
    ok = lines[:4] + ["v_add_u32_e32 v2, v1, v3"] + lines[5:]
    assert scan(ok)[1] == {}


@pytest.mark.skipif(shutil.which("hipcc") is None and not os.path.exists("/opt/rocm/bin/hipcc"),
                    reason="hipcc not available")
def test_inline_lds_reads_are_not_touched_before_their_wait(tmp_path):
    from paper_2301_09830_amd import build
    cmd = build.compile_command(str(tmp_path / "api.s"))
    cmd = [c for c in cmd if c not in ("-fPIC", "-shared")] + ["--cuda-device-only", "-S"]
    proc = subprocess.run(cmd, capture_output=True, text=True)
    assert proc.returncode == 0, proc.stderr[-2000:]
    kernels, bad = scan(open(tmp_path / "api.s").read().split("\n"))
    # the rank-16 left product, the fp32 and bf16 right products use them
    assert any("k_pm" in k for k in kernels) and any("k_lq" in k for k in kernels)
    assert any("k_lqx" in k for k in kernels)
    assert bad == {}, f"instructions touch in-flight LDS read registers: {bad}"
