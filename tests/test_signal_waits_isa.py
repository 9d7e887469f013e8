"""The slot signals and producer waits in the built kernels' machine code (CPU only).

A consumer releases a slot with `s_waitcnt lgkmcnt(n)` followed by
`ds_add_u32`, where n counts the LDS reads issued after the last read of the
slot.  LDS operations complete in issue order, scalar-memory loads
(s_load, s_buffer_load, s_memtime, s_memrealtime) share the counter and may
complete out of order.  tests/test_lgkm_counting.py shows on a model of the
counter that a scalar load in flight never weakens such a wait; this test
checks the stronger property on the compiled code itself, so that the
release does not depend on that argument at all: at every `ds_add_u32` whose
nearest wait is lgkmcnt(n) with n > 0, no scalar load may still be in flight
on any path into that wait (a scalar load is known complete only after an
lgkmcnt(0) wait).  A second check covers the register-staged producers'
global-load waits: the wait before a slot write never drains the loads of the
K-iterations staged behind it.

The code is read from the gfx950 code objects of paper_2506_11209_amd/
libwsgemm.so (built here from source) and disassembled with the ROCm
toolchain's llvm-objdump; the analysis is a forward may-analysis over the
control-flow graph of each kernel (branch targets as printed by the
disassembler).
"""
import os
import re
import subprocess
import tempfile

import pytest

from paper_2506_11209_amd import kernel_code as kc

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIB = os.path.join(ROOT, "paper_2506_11209_amd", "libwsgemm.so")
OBJDUMP = "/opt/rocm/llvm/bin/llvm-objdump"

SCALAR_LOADS = ("s_load", "s_buffer_load", "s_memtime", "s_memrealtime")
_FN = re.compile(r"^([0-9a-f]+) <(\S+)>:$")
_INS = re.compile(r"^\s+(\S+)(.*?)//\s*([0-9A-F]+):[^<]*(?:<(\S+)\+0x([0-9a-f]+)>)?")
_LGKM = re.compile(r"lgkmcnt\((\d+)\)")


def lgkm_of(operands: str):
    m = _LGKM.search(operands)
    return int(m.group(1)) if m else None


def disassemble(code_object: bytes) -> dict:
    """{kernel: (start address, [(address, mnemonic, operands, branch target offset or None)])}."""
    with tempfile.NamedTemporaryFile(suffix=".o", delete=False) as f:
        f.write(code_object)
        path = f.name
    try:
        out = subprocess.run([OBJDUMP, "-d", "--mcpu=gfx950", path], capture_output=True, text=True,
                             check=True).stdout
    finally:
        os.unlink(path)
    fns, cur = {}, None
    for line in out.splitlines():
        m = _FN.match(line)
        if m:
            cur = []
            fns[m.group(2)] = (int(m.group(1), 16), cur)
            continue
        m = _INS.match(line)
        if m and cur is not None:
            tgt = int(m.group(5), 16) if m.group(4) else None
            cur.append((int(m.group(3), 16), m.group(1), m.group(2).strip(), tgt))
    return fns


def successors(start: int, ins: list) -> list:
    index = {a: i for i, (a, _, _, _) in enumerate(ins)}
    succ = [[] for _ in ins]
    for i, (a, mn, _, tgt) in enumerate(ins):
        if mn in ("s_endpgm", "s_trap") or mn.startswith("s_setpc"):
            continue
        if mn.startswith(("s_branch", "s_cbranch")):
            assert tgt is not None and start + tgt in index, (hex(a), mn)
            succ[i].append(index[start + tgt])
            if mn.startswith("s_cbranch") and i + 1 < len(ins):
                succ[i].append(i + 1)
        elif i + 1 < len(ins):
            succ[i].append(i + 1)
    return succ


def unsafe_signals(start: int, ins: list):
    """(signals checked, [(address, reason)]) for one kernel."""
    succ = successors(start, ins)
    pending = [False] * len(ins)  # before instruction i: a scalar load may be in flight
    reached = [False] * len(ins)
    if ins:
        reached[0] = True
    work = [0] if ins else []
    while work:
        i = work.pop()
        s = pending[i]
        _, mn, ops, _ = ins[i]
        if mn.startswith(SCALAR_LOADS):
            s = True
        elif mn == "s_waitcnt" and lgkm_of(ops) == 0:
            s = False
        for j in succ[i]:
            if not reached[j] or (s and not pending[j]):
                reached[j] = True
                pending[j] = pending[j] or s
                work.append(j)
    bad, checked = [], 0
    for i, (a, mn, _, _) in enumerate(ins):
        if not mn.startswith("ds_add") or not reached[i]:
            continue
        j = i - 1  # the wait guarding this signal: straight-line code before it
        while j >= 0 and not (ins[j][1] == "s_waitcnt" and lgkm_of(ins[j][2]) is not None):
            if ins[j][1].startswith(("s_branch", "s_cbranch", "ds_") + SCALAR_LOADS):
                j = -1
                break
            j -= 1
        if j < 0:
            bad.append((hex(a), "no LDS wait before the signal"))
            continue
        checked += 1
        n = lgkm_of(ins[j][2])
        if n > 0 and pending[j]:
            bad.append((hex(a), "lgkmcnt(%d) with a scalar load in flight" % n))
    return checked, bad


def _ins(*rows):
    return [(4 * k, mn, ops, tgt) for k, (mn, ops, tgt) in enumerate(rows)]


def test_the_analysis_flags_a_scalar_load_in_flight():
    ok = _ins(("s_load_dword", "s4, s[0:1], 0x0", None), ("s_waitcnt", "lgkmcnt(0)", None),
              ("ds_read_b128", "v[0:3], v8", None), ("ds_read_b128", "v[4:7], v9", None),
              ("s_waitcnt", "lgkmcnt(1)", None), ("s_mov_b64", "s[2:3], exec", None),
              ("ds_add_u32", "v10, v11", None), ("s_endpgm", "", None))
    assert unsafe_signals(0, ok) == (1, [])
    planted = _ins(("ds_read_b128", "v[0:3], v8", None), ("s_load_dword", "s4, s[0:1], 0x0", None),
                   ("ds_read_b128", "v[4:7], v9", None), ("s_waitcnt", "lgkmcnt(1)", None),
                   ("ds_add_u32", "v10, v11", None), ("s_endpgm", "", None))
    checked, bad = unsafe_signals(0, planted)
    assert checked == 1 and len(bad) == 1 and "in flight" in bad[0][1]
    # a scalar load issued late in a loop body reaches the signal at the loop top
    loop = _ins(("ds_read_b128", "v[0:3], v8", None), ("s_waitcnt", "lgkmcnt(1)", None),
                ("ds_add_u32", "v10, v11", None), ("s_memtime", "s[4:5]", None),
                ("s_cbranch_scc1", "-5", 0), ("s_endpgm", "", None))
    assert len(unsafe_signals(0, loop)[1]) == 1
    # lgkmcnt(0) is always safe; a signal with no wait is reported
    drained = _ins(("s_load_dword", "s4, s[0:1], 0x0", None), ("s_waitcnt", "vmcnt(0) lgkmcnt(0)", None),
                   ("ds_add_u32", "v10, v11", None), ("s_endpgm", "", None))
    assert unsafe_signals(0, drained) == (1, [])
    unguarded = _ins(("ds_read_b128", "v[0:3], v8", None), ("ds_add_u32", "v10, v11", None),
                     ("s_endpgm", "", None))
    assert unsafe_signals(0, unguarded)[1][0][1] == "no LDS wait before the signal"


_needs_lib = [pytest.mark.skipif(not os.path.exists(LIB), reason="library not built"),
              pytest.mark.skipif(not os.path.exists(OBJDUMP), reason="llvm-objdump not found")]


@pytest.fixture(scope="module")
def library_code():
    """[(kernel, start, instructions)] of every kernel in the built library."""
    with open(LIB, "rb") as f:
        lib = f.read()
    return [(name, start, ins) for co in kc._code_objects(lib) for name, (start, ins) in disassemble(co).items()]


@_needs_lib[0]
@_needs_lib[1]
def test_no_signal_waits_on_a_count_that_a_scalar_load_shares(library_code):
    kernels = signals = younger = 0
    problems = []
    for name, start, ins in library_code:
        checked, bad = unsafe_signals(start, ins)
        kernels += 1
        signals += checked
        younger += sum(1 for (_, mn, ops, _) in ins if mn == "s_waitcnt" and (lgkm_of(ops) or 0) > 0)
        problems += [(name, a, why) for a, why in bad]
    assert kernels > 400 and signals > 1000 and younger > 0
    assert not problems, problems[:10]


def staged_write_waits(ins):
    """vmcnt of the wait guarding each ds_write_b128 (the register-staged
    producers' slot writes), in program order."""
    out = []
    for i, (_, mn, _, _) in enumerate(ins):
        if mn != "ds_write_b128":
            continue
        j = i - 1
        while j >= 0 and ins[j][1] != "s_waitcnt" and not ins[j][1].startswith("ds_write"):
            j -= 1
        if j >= 0 and ins[j][1] == "s_waitcnt":
            m = re.search(r"vmcnt\((\d+)\)", ins[j][2])
            if m:
                out.append(int(m.group(1)))
    return out


@_needs_lib[0]
@_needs_lib[1]
def test_register_staged_producers_never_drain_their_staged_loads(library_code):
    """A register-staged producer keeps several K-iterations of loads in
    flight and writes the oldest one to its slot: the wait before that write
    must leave the newer iterations' loads outstanding.  A wait for every
    load (vmcnt(0)) there empties the pipeline and exposes a full memory
    latency.  The compiler placed one at the first register stage of every
    pass through the stages while the wait loop could leave the loop early
    (10 % of the load-only time at 16384 x 256 x 8192), and before every
    slot write of the general variant while its loads branched between an
    interior and an edge form (8000^3 ran at a third of its speed)."""
    kernels, drained = 0, []
    for name, _, ins in library_code:
        if "ws_gemm_kernel" not in name:
            continue
        waits = staged_write_waits(ins)
        if waits:
            kernels += 1
            if min(waits) == 0:
                drained.append((name, waits[:16]))
    assert kernels > 300
    assert not drained, drained[:5]
