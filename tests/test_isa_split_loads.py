"""The decode kernel's split K/V loads are issued as inline assembly, which the
compiler's wait counting does not see (the K/V tile, query and range-end
counter loads): the kernel must not read or write a load's destination
registers before its own explicit wait.  This compiles
the stream-K kernels for gfx950 to assembly (no GPU needed) and checks, for
every inline-assembly load of every matrix-core instantiation, that no
instruction between the load and the next `s_waitcnt vmcnt` (in program text
order) names one of its destination registers.  A compiler that copied such
a register early (a value not yet arrived) would fail here, not silently on
the GPU."""
import importlib.util
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
_spec = importlib.util.spec_from_file_location("pa_build", os.path.join(ROOT, "paper_2504_09345_amd", "build.py"))
build = importlib.util.module_from_spec(_spec)  # the library's own build flags
_spec.loader.exec_module(build)


def _regs(text):
    out = set()
    for m in re.finditer(r"\bv\[(\d+):(\d+)\]", text):
        out |= set(range(int(m.group(1)), int(m.group(2)) + 1))
    for m in re.finditer(r"\bv(\d+)\b", text):
        out.add(int(m.group(1)))
    return out


def _kernels(asm):
    """(name, instruction lines, indexes of the inline-assembly loads) of each
    stream-K kernel with the matrix-core fold (template argument MF = true:
    `...ELb1ELb0E...` or `...ELb1ELb1E...`).  Inline assembly sits between
    `;;#ASMSTART` and `;;#ASMEND` in the compiler's output."""
    out = []
    for m in re.finditer(r"^(_ZN2pa13stream_kernel\w+):", asm, flags=re.M):
        name = m.group(1)
        if not re.search(r"Li2ELb1ELb[01]E", name):
            continue
        end = asm.index(".Lfunc_end", m.end())
        lines, loads, in_asm = [], [], False
        for l in (l.strip() for l in asm[m.end():end].splitlines()):
            if l.startswith(";;#ASMSTART"):
                in_asm = True
            elif l.startswith(";;#ASMEND"):
                in_asm = False
            elif l and not l.startswith(";"):
                if in_asm and re.match(r"(buffer|global)_load_", l):
                    loads.append(len(lines))
                lines.append(l)
        out.append((name, lines, loads))
    return out


@pytest.fixture(scope="module", params=["pa_stream.hip", "pa_trace.hip"])
def stream_asm(request, tmp_path_factory):
    """The production stream-K kernels and their gather-trace instantiations
    (which the bit-exact gather test runs)."""
    if not os.path.exists(build.HIPCC):
        pytest.skip("hipcc not available")
    out = tmp_path_factory.mktemp("isa") / (request.param + ".s")
    cmd = [build.HIPCC, *build.FLAGS, "--cuda-device-only", "-S",
           os.path.join(build.CSRC, request.param), "-o", str(out)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    return open(out).read()


_VM_OP = re.compile(r"(buffer|global|flat|scratch)_(load|store|atomic)")
_BRANCH = re.compile(r"s_(c?branch)\w*\s+(\.LBB\w+)")


def _untouched(lines, labels, loads, i, dst, counted=True):
    """Follow every control-flow path from the load at line i until a wait
    retires it and return the first line on the way that names a register of
    dst, else None.  counted: a wait retires the load when it is `s_waitcnt
    vmcnt(N)` with at least N vector-memory operations issued after the load
    on that path (they retire in issue order); else any `s_waitcnt vmcnt`
    ends the path."""
    todo, seen = [(i + 1, 0)], set()
    while todo:
        j, younger = todo.pop()
        while j < len(lines):
            if (j, younger) in seen:
                break
            seen.add((j, younger))
            t = lines[j]
            m = re.match(r"s_waitcnt\b.*vmcnt\((\d+)\)", t)
            if m and (younger >= int(m.group(1)) or not counted):
                break  # retired on this path
            if t.startswith("s_endpgm"):
                break
            if not t.startswith(".") and j not in loads and _regs(t) & dst:
                return t
            if _VM_OP.match(t):
                younger = min(younger + 1, 64)
            b = _BRANCH.match(t)
            if b:
                target = labels[b.group(2)]
                if b.group(1) == "branch":
                    j = target
                    continue
                todo.append((target, younger))
            j += 1
    return None


def test_split_loads_are_untouched_until_their_wait(stream_asm):
    kernels = _kernels(stream_asm)
    assert kernels, "no matrix-core stream-K kernel in the assembly"
    checked = 0
    counter_loads = 0
    for name, lines, loads in kernels:
        assert loads, f"{name}: no inline-assembly loads (split K/V schedule not compiled in)"
        counter_loads += sum(lines[i].startswith("global_load_dwordx2") for i in loads)
        labels = {m.group(1): j for j, l in enumerate(lines) if (m := re.match(r"(\.LBB\w+):", l))}
        loads = set(loads)
        for i in sorted(loads):
            m = re.match(r"\w+ v\[(\d+):(\d+)\]", lines[i])
            dst = set(range(int(m.group(1)), int(m.group(2)) + 1))
            # The range-end counter is loaded a unit before the unit that
            # reads it; the static paths also run from its load straight into
            # that read within one iteration (the unit index rules that out),
            # so for it any wait ends a path; the tile and query loads are
            # checked with the wait counts.
            t = _untouched(lines, labels, loads, i, dst, counted=not lines[i].startswith("global_load"))
            assert t is None, f"{name}: `{t}` touches {lines[i]!r} before its wait"
            checked += 1
    assert checked >= 20
    # the range-end counter load of every instantiation (before the loop and in it)
    assert counter_loads >= 2 * len(kernels)


def _check(text):
    """_untouched over a hand-written instruction list: the first offending
    line for each inline-assembly load (lines marked with a leading '*')."""
    lines, loads = [], set()
    for l in text.strip().splitlines():
        l = l.strip()
        if l.startswith("*"):
            loads.add(len(lines))
            l = l[1:].strip()
        lines.append(l)
    labels = {m.group(1): j for j, l in enumerate(lines) if (m := re.match(r"(\.LBB\w+):", l))}
    out = []
    for i in sorted(loads):
        m = re.match(r"\w+ v\[(\d+):(\d+)\]", lines[i])
        out.append(_untouched(lines, labels, loads, i, set(range(int(m.group(1)), int(m.group(2)) + 1))))
    return out


def test_checker_on_hand_written_paths():
    # a use after a wait that retires the load passes; one before it fails
    assert _check("""
        *buffer_load_dwordx4 v[4:7], v1, s[0:3], 0 offen offset:0 nt
        s_waitcnt vmcnt(0)
        v_add_f32_e32 v8, v4, v5
        s_endpgm""") == [None]
    assert _check("""
        *buffer_load_dwordx4 v[4:7], v1, s[0:3], 0 offen offset:0 nt
        v_mov_b32_e32 v6, 0
        s_waitcnt vmcnt(0)
        s_endpgm""") == ["v_mov_b32_e32 v6, 0"]
    # vmcnt(1) retires the older of two loads only
    assert _check("""
        *buffer_load_dwordx4 v[4:7], v1, s[0:3], 0 offen offset:0 nt
        *buffer_load_dwordx4 v[8:11], v1, s[0:3], 0 offen offset:64 nt
        s_waitcnt vmcnt(1)
        v_add_f32_e32 v12, v4, v8
        s_endpgm""") == [None, "v_add_f32_e32 v12, v4, v8"]
    # a branch around the wait reaches the use
    assert _check("""
        *buffer_load_dwordx4 v[4:7], v1, s[0:3], 0 offen offset:0 nt
        s_cbranch_scc1 .LBB0_2
        s_waitcnt vmcnt(0)
        .LBB0_2:
        v_add_f32_e32 v12, v4, v4
        s_endpgm""") == ["v_add_f32_e32 v12, v4, v4"]
    # an unconditional branch skips the lines after it
    assert _check("""
        *buffer_load_dwordx4 v[4:7], v1, s[0:3], 0 offen offset:0 nt
        s_branch .LBB0_3
        v_mov_b32_e32 v4, 0
        .LBB0_3:
        s_waitcnt vmcnt(0)
        v_mov_b32_e32 v4, 0
        s_endpgm""") == [None]
