"""Checks on the gfx950 assembly of the library's tile loops (built here,
host only, no GPU).

1. The tile loops issue some LDS reads as inline assembly (so that the
   compiler does not wait for DMA into other stages) and end each batch with
   an s_waitcnt lgkmcnt(0) that names the read values as operands.  Until that
   wait a read's destination registers are still being written by the LDS, so
   no compiler-generated instruction may touch them in between.

2. The same loops wait for their LDS DMA with hand-written
   s_waitcnt vmcnt(N) immediates, counted from the number of load
   instructions one stage issues.  Vector-memory instructions complete in
   order, so the wait is right only if N equals what the loop really issues
   after the stage it needs.  The scan builds each kernel's control-flow
   graph, takes the loop (strongly connected component) holding each
   hand-written wait, counts the vector-memory instructions in it (c per
   iteration) and requires: the left product at rank <= 16 and the fp32
   right product wait for {0, c, 2c} (zero, one or two later stages still in
   flight); the bf16 rank-128 right product waits for c minus the wave's share
   of the P-tile loads (the A tile issued after them is all that may remain).
   A spill or an extra load inside a loop changes c and fails the check."""

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


HAVE_HIPCC = shutil.which("hipcc") is not None or os.path.exists("/opt/rocm/bin/hipcc")


@pytest.fixture(scope="module")
def asm_lines(tmp_path_factory):
    from paper_2301_09830_amd import build
    out = tmp_path_factory.mktemp("asm") / "api.s"
    cmd = build.compile_command(str(out))
    cmd = [c for c in cmd if c not in ("-fPIC", "-shared")] + ["--cuda-device-only", "-S"]
    proc = subprocess.run(cmd, capture_output=True, text=True)
    assert proc.returncode == 0, proc.stderr[-2000:]
    return open(out).read().split("\n")


@pytest.mark.skipif(not HAVE_HIPCC, reason="hipcc not available")
def test_inline_lds_reads_are_not_touched_before_their_wait(asm_lines):
    kernels, bad = scan(asm_lines)
    # the rank-16 left product, the fp32 and bf16 right products use them
    assert any("k_pm" in k for k in kernels) and any("k_lq" in k for k in kernels)
    assert any("k_lqx" in k for k in kernels)
    assert bad == {}, f"instructions touch in-flight LDS read registers: {bad}"


# ---------------------------------------------------------------------------
# hand-written vmcnt waits against the loads the loops issue
# ---------------------------------------------------------------------------
VMEM = re.compile(r"^(global_|buffer_|flat_|scratch_)")
BRANCH = re.compile(r"^s_(c?)branch\S*\s+(\.LBB\d+_\d+)")


def functions(lines):
    funcs, cur = {}, None
    for line in lines:
        m = re.match(r"^(_Z\S+):", line)
        if m:
            cur = m.group(1)
            funcs[cur] = []
            continue
        if cur is not None:
            if line.startswith(".Lfunc_end"):
                cur = None
                continue
            funcs[cur].append(line)
    return funcs


def basic_blocks(body):
    """[(label, instructions)] and successor lists of one function."""
    blocks, cur = [], [None, []]
    for line in body:
        t = line.strip()
        m = re.match(r"^(\.LBB\d+_\d+):", t)
        if m:
            blocks.append(cur)
            cur = [m.group(1), []]
            continue
        if not t.startswith(";;#"):
            t = t.split(";")[0].strip()
        if not t or t.startswith("."):
            continue
        cur[1].append(t)
        if t.startswith(("s_branch", "s_cbranch", "s_endpgm", "s_setpc")):
            blocks.append(cur)
            cur = [None, []]
    blocks.append(cur)
    blocks = [b for b in blocks if b[0] is not None or b[1]]
    where = {b[0]: i for i, b in enumerate(blocks) if b[0]}
    succ = []
    for i, (_, ins) in enumerate(blocks):
        last = ins[-1] if ins else ""
        m = BRANCH.match(last)
        s = []
        if m:
            s.append(where[m.group(2)])
            if m.group(1) == "c" and i + 1 < len(blocks):
                s.append(i + 1)
        elif not last.startswith(("s_endpgm", "s_setpc")) and i + 1 < len(blocks):
            s.append(i + 1)
        succ.append(s)
    return blocks, succ


def strongly_connected(n, succ):
    """Tarjan's algorithm, iterative."""
    index, low, on, stack, comps = {}, {}, set(), [], []
    counter = 0
    for root in range(n):
        if root in index:
            continue
        work = [(root, 0)]
        while work:
            v, k = work.pop()
            if k == 0:
                index[v] = low[v] = counter
                counter += 1
                stack.append(v)
                on.add(v)
            if k < len(succ[v]):
                work.append((v, k + 1))
                w = succ[v][k]
                if w not in index:
                    work.append((w, 0))
                elif w in on:
                    low[v] = min(low[v], index[w])
                continue
            if low[v] == index[v]:
                comp = []
                while True:
                    w = stack.pop()
                    on.discard(w)
                    comp.append(w)
                    if w == v:
                        break
                comps.append(comp)
            if work:
                u = work[-1][0]
                low[u] = min(low[u], low[v])
    return comps


def loops(blocks_in, succ, preds):
    """Every loop of the control-flow graph restricted to `blocks_in`, nested
    loops included: each nontrivial strongly connected component, then,
    with the edges back into its header removed (the block entered from
    outside it, else its first block), the loops inside it."""
    idx = sorted(blocks_in)
    pos = {b: i for i, b in enumerate(idx)}
    sub = [[pos[w] for w in succ[b] if w in pos] for b in idx]
    out = []
    for comp in strongly_connected(len(idx), sub):
        members = {idx[i] for i in comp}
        if len(members) == 1:
            b = next(iter(members))
            if b not in succ[b]:
                continue
        out.append(members)
        entries = [b for b in members if any(p not in members for p in preds[b])]
        header = min(entries) if entries else min(members)
        inner_succ = {b: [w for w in succ[b] if w != header] for b in members}
        full = [inner_succ.get(b, []) for b in range(len(succ))]
        out.extend(loops(members - {header}, full, preds))
    return out


def loop_waits(body):
    """For each innermost loop holding hand-written vmcnt waits: (waits,
    vector-memory instructions per iteration)."""
    blocks, succ = basic_blocks(body)
    preds = [[] for _ in blocks]
    for v, ws in enumerate(succ):
        for w in ws:
            preds[w].append(v)

    def waits_of(members):
        found = set()
        for b in members:
            ins = blocks[b][1]
            for j, t in enumerate(ins):
                m = re.match(r"s_waitcnt vmcnt\((\d+)\)$", t)
                if m and j > 0 and ins[j - 1].startswith(";;#ASMSTART"):
                    found.add(int(m.group(1)))
        return found

    with_waits = [c for c in loops(set(range(len(blocks))), succ, preds) if any(waits_of(c))]
    out = []
    for c in with_waits:
        if any(o < c and waits_of(o) == waits_of(c) for o in with_waits):
            continue   # a loop nested in this one holds the same waits
        out.append((sorted(waits_of(c)), sum(1 for b in c for t in blocks[b][1] if VMEM.match(t))))
    return out


def wait_violations(funcs):
    """(kernels checked, problems).  Stage loops wait for {0, c, 2c}; the bf16
    rank-RP right product for c minus its P-tile share ceil(2 (RP / 32) / W),
    W its waves per block (8 at rank 128, else 4)."""
    checked, bad = set(), []
    for name, body in funcs.items():
        for waits, c in loop_waits(body):
            checked.add(name)
            if "k_lqx" in name:
                rp = int(re.search(r"k_lqxILi\d+ELi(\d+)E", name).group(1))
                share = -(-2 * (rp // 32) // (8 if rp >= 128 else 4))
                want = [0, c - share]
            elif "k_pm" in name or "k_lq" in name:
                want = [0, c, 2 * c]
            else:
                bad.append((name, "unknown loop with hand-written vmcnt waits", waits, c))
                continue
            # a loop may hold only some of them (the compiler peels or
            # versions the stage loop), never another value
            if not set(waits) <= set(want) or c <= 0 or want[1] <= 0:
                bad.append((name, waits, c, want))
    return checked, bad


def test_wait_scan_flags_a_drifted_count():
    """A loop that issues 3 loads per stage but waits as if it issued 4."""
    good = ["_ZN3occ4k_pmXE:", ".LBB0_1:", "global_load_lds_dwordx4 v[2:3], off",
            "global_load_lds_dwordx4 v[2:3], off", "global_load_lds_dwordx4 v[2:3], off",
            ";;#ASMSTART", "s_waitcnt vmcnt(6)", ";;#ASMEND", ";;#ASMSTART", "s_waitcnt vmcnt(3)",
            ";;#ASMEND", ";;#ASMSTART", "s_waitcnt vmcnt(0)", ";;#ASMEND",
            "s_cbranch_scc1 .LBB0_1", "s_endpgm", ".Lfunc_end0:"]
    checked, bad = wait_violations(functions(good))
    assert checked == {"_ZN3occ4k_pmXE"} and bad == []
    drifted = [ln.replace("vmcnt(6)", "vmcnt(8)").replace("vmcnt(3)", "vmcnt(4)") for ln in good]
    assert wait_violations(functions(drifted))[1]
    spilled = good[:2] + ["scratch_load_dword v9, off, s32"] + good[2:]
    assert wait_violations(functions(spilled))[1]
    # the same loop nested in an outer loop that issues other loads: the
    # inner loop is the one checked
    nested = (good[:1] + [".LBB0_0:", "global_load_dwordx4 v[4:7], v[2:3], off"] + good[1:-2]
              + ["global_store_dword v[2:3], v4, off", "s_cbranch_scc1 .LBB0_0", "s_endpgm", ".Lfunc_end0:"])
    assert wait_violations(functions(nested)) == ({"_ZN3occ4k_pmXE"}, [])
    nested_drifted = [ln.replace("vmcnt(6)", "vmcnt(8)").replace("vmcnt(3)", "vmcnt(4)") for ln in nested]
    assert wait_violations(functions(nested_drifted))[1]


@pytest.mark.skipif(not HAVE_HIPCC, reason="hipcc not available")
def test_vmcnt_waits_match_the_loads_each_loop_issues(asm_lines):
    checked, bad = wait_violations(functions(asm_lines))
    assert any("k_pm" in k for k in checked) and any("k_lqx" in k for k in checked)
    assert any("k_lq" in k and "k_lqx" not in k for k in checked)
    assert bad == [], f"hand-written vmcnt waits disagree with the loads issued: {bad}"
