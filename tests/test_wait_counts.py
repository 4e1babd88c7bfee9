"""The hand-counted vector-memory waits of the kernels, checked on their compiled gfx950 code,
and the wait states ahead of their direct-to-LDS loads.

The token, convolution and attention kernels stage weights and K/V with direct global->LDS
loads and await them with `s_waitcnt vmcnt(N)`, where N counts the vector memory operations
the wavefront issued after its newest direct load (operations retire in issue order). A wrong
N leaves a load in flight when the workgroup barrier publishes the buffer, or when the
workgroup ends and its LDS is handed to the next one. This test disassembles the library's own
build (the gfx950 code object inside each object file of paper_2601_09921_amd/_build) and
runs a dataflow over every kernel's control-flow graph: per program point, the fewest vector
memory operations issued since the newest direct-to-LDS load on any path into it. A wait
vmcnt(k) completes that load iff the count is >= k. At every s_barrier and s_endpgm no direct
load may remain possibly pending.

The direct loads are inline assembly, so the compiler inserts no wait states for their operands.
A vector instruction that writes an SGPR must be followed by 5 wait states before a vector
memory instruction reads that SGPR (the load address), or the load reads the register's old
value -- a load from the wrong address. Every direct load must therefore sit at least 5 wait
states after the last vector write of its address registers on the straight-line path before it.
"""
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
OBJDIR = os.path.join(ROOT, "paper_2601_09921_amd", "_build")
LLVM = "/opt/rocm/llvm/bin"
TARGET = "hipv4-amdgcn-amd-amdhsa--gfx950"
INF = 1 << 30
VMEM = re.compile(r"^(global_|buffer_|scratch_|flat_)")
DMA = re.compile(r"^global_load_lds_")
VMCNT = re.compile(r"^s_waitcnt\b.*\bvmcnt\((\d+)\)")
LINE = re.compile(r"^\s+(\S+)(.*?)//\s*([0-9A-F]+):")
FUNC = re.compile(r"^([0-9a-f]+) <(\w+)>:$")
TARGET_RE = re.compile(r"<(\w+)\+0x([0-9a-f]+)>")


def disassemble(obj: str, tmp) -> str:
    fat = tmp / (os.path.basename(obj) + ".fatbin")
    co = tmp / (os.path.basename(obj) + ".co")
    subprocess.run([f"{LLVM}/llvm-objcopy", f"--dump-section=.hip_fatbin={fat}", obj, str(tmp / "discard.o")],
                   check=True, capture_output=True)
    subprocess.run([f"{LLVM}/clang-offload-bundler", "--unbundle", "--type=o", f"--targets={TARGET}",
                    f"--input={fat}", f"--output={co}"], check=True, capture_output=True)
    return subprocess.run([f"{LLVM}/llvm-objdump", "-d", "--mcpu=gfx950", str(co)], check=True,
                          capture_output=True, text=True).stdout


def functions(text: str):
    """{name: [(address, mnemonic, operands, branch target or None)]}"""
    funcs, cur, base = {}, None, {}
    for ln in text.splitlines():
        m = FUNC.match(ln)
        if m:
            cur = m.group(2)
            base[cur] = int(m.group(1), 16)
            funcs[cur] = []
            continue
        m = LINE.match(ln)
        if cur and m:
            t = TARGET_RE.search(ln)
            tgt = base[t.group(1)] + int(t.group(2), 16) if t and t.group(1) in base else None
            funcs[cur].append((int(m.group(3), 16), m.group(1), m.group(2).strip(), tgt))
    return funcs


def check(insts) -> list[str]:
    """Places where a direct-to-LDS load may still be pending at a barrier or at the end."""
    idx = {a: i for i, (a, *_) in enumerate(insts)}
    # successors of each instruction
    def succ(i):
        a, mn, _, tgt = insts[i]
        if mn == "s_endpgm":
            return []
        if mn == "s_branch":
            return [idx[tgt]]
        out = [i + 1] if i + 1 < len(insts) else []
        if mn.startswith("s_cbranch") and tgt in idx:
            out.append(idx[tgt])
        return out
    state = [None] * len(insts)
    state[0] = INF
    work = [0]
    problems = []
    while work:
        i = work.pop()
        st = state[i]
        _, mn, ops, _ = insts[i]
        if DMA.match(mn):
            st = 0
        elif VMEM.match(mn):
            st = st + 1 if st < INF else INF
        else:
            m = VMCNT.match(mn + " " + ops)
            if m and st >= int(m.group(1)):
                st = INF
        for j in succ(i):
            if state[j] is None or st < state[j]:
                state[j] = st
                work.append(j)
    for i, (a, mn, ops, _) in enumerate(insts):
        if mn in ("s_barrier", "s_endpgm") and state[i] is not None and state[i] < INF:
            problems.append(f"{mn} at 0x{a:x} with a direct LDS load possibly pending ({state[i]} ops after it)")
    return problems


SREG = re.compile(r"^s\[(\d+):(\d+)\]$|^s(\d+)$")


def sregs(tok: str) -> set:
    m = SREG.match(tok.strip().rstrip(","))
    if not m:
        return set()
    if m.group(3) is not None:
        return {int(m.group(3))}
    return set(range(int(m.group(1)), int(m.group(2)) + 1))


def sgpr_hazards(insts, need_states: int = 5) -> list[str]:
    """Direct-to-LDS loads closer than need_states wait states to a vector write of one of
    their SGPR operands (scanning back along the instruction stream)."""
    problems = []
    for i, (a, mn, ops, _) in enumerate(insts):
        if not DMA.match(mn):
            continue
        need = set()
        for t in ops.split(",")[1:]:
            if t.strip():
                need |= sregs(t.split()[0])
        states = 0
        for j in range(i - 1, max(i - 16, -1), -1):
            _, pm, pops, _ = insts[j]
            if pm == "s_nop":
                states += int(pops.split()[0]) + 1
                continue
            if states >= need_states:
                break
            if pm.startswith("v_") and pops and sregs(pops.split(",")[0]) & need:
                problems.append(f"{pm} {pops} at {states} wait states before {mn} {ops} at 0x{a:x}")
                break
            states += 1
    return problems


def objects():
    if not os.path.isdir(OBJDIR):
        return []
    return sorted(os.path.join(OBJDIR, f) for f in os.listdir(OBJDIR) if f.endswith(".hip.o"))


@pytest.mark.parametrize("obj", objects(), ids=[os.path.basename(o) for o in objects()])
def test_direct_lds_loads_complete_before_barriers(obj, tmp_path):
    if not os.path.exists(f"{LLVM}/llvm-objdump"):
        pytest.skip("ROCm LLVM tools not found")
    funcs = functions(disassemble(obj, tmp_path))
    assert funcs, "no kernels found"
    if os.path.basename(obj) in ("tok.hip.o", "attn.hip.o", "resident.hip.o"):   # these stage through direct loads
        assert any(DMA.match(mn) for insts in funcs.values() for _, mn, _, _ in insts)
    bad = {name: p for name, insts in funcs.items() if (p := check(insts))}
    assert not bad, bad


@pytest.mark.parametrize("obj", objects(), ids=[os.path.basename(o) for o in objects()])
def test_direct_lds_load_addresses_are_settled(obj, tmp_path):
    if not os.path.exists(f"{LLVM}/llvm-objdump"):
        pytest.skip("ROCm LLVM tools not found")
    funcs = functions(disassemble(obj, tmp_path))
    bad = {name: p for name, insts in funcs.items() if (p := sgpr_hazards(insts))}
    assert not bad, bad


def test_the_address_check_catches_a_fresh_sgpr():
    """A planted mistake: the load's address register written by v_readfirstlane just before."""
    insts = [(0, "v_readfirstlane_b32", "s20, v144", None), (4, "v_readfirstlane_b32", "s21, v145", None),
             (8, "global_load_lds_dwordx4", "v98, s[20:21]", None)]
    assert sgpr_hazards(insts)
    insts.insert(2, (6, "s_nop", "4", None))
    assert not sgpr_hazards(insts)


def test_the_check_catches_a_missing_wait():
    """A planted mistake: a direct load followed by one store and a wait that allows one op
    in flight before a barrier -- the load may still be pending there."""
    insts = [(0, "global_load_lds_dwordx4", "v1, s[0:1]", None), (4, "global_store_dwordx4", "v[0:1], v[2:5], off", None),
             (8, "s_waitcnt", "vmcnt(2)", None), (12, "s_barrier", "", None), (16, "s_endpgm", "", None)]
    assert check(insts)
    insts[2] = (8, "s_waitcnt", "vmcnt(1)", None)
    assert not check(insts)
