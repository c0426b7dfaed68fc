"""The decode kernel's split K/V loads are issued as inline assembly, which the
compiler's wait counting does not see: the kernel must not read or write a
load's destination registers before its own explicit wait.  This compiles
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
    """(name, instruction lines) of each stream-K kernel with the matrix-core
    fold (template argument MF = true: `...ELb1ELb0E...` or `...ELb1ELb1E...`)."""
    out = []
    for m in re.finditer(r"^(_ZN2pa13stream_kernel\w+):", asm, flags=re.M):
        name = m.group(1)
        if not re.search(r"Li2ELb1ELb[01]E", name):
            continue
        end = asm.index(".Lfunc_end", m.end())
        body = [l.strip() for l in asm[m.end():end].splitlines()]
        out.append((name, [l for l in body if l and not l.startswith(";")]))
    return out


@pytest.fixture(scope="module")
def stream_asm(tmp_path_factory):
    if not os.path.exists(build.HIPCC):
        pytest.skip("hipcc not available")
    out = tmp_path_factory.mktemp("isa") / "pa_stream.s"
    cmd = [build.HIPCC, *build.FLAGS, "--cuda-device-only", "-S",
           os.path.join(build.CSRC, "pa_stream.hip"), "-o", str(out)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    return open(out).read()


def test_split_loads_are_untouched_until_their_wait(stream_asm):
    kernels = _kernels(stream_asm)
    assert kernels, "no matrix-core stream-K kernel in the assembly"
    checked = 0
    for name, lines in kernels:
        loads = [i for i, l in enumerate(lines) if l.startswith("buffer_load_dwordx4") and "offen offset:" in l]
        assert loads, f"{name}: no inline-assembly loads (split K/V schedule not compiled in)"
        for i in loads:
            m = re.match(r"buffer_load_dwordx4 v\[(\d+):(\d+)\]", lines[i])
            dst = set(range(int(m.group(1)), int(m.group(2)) + 1))
            for j in range(i + 1, len(lines)):
                t = lines[j]
                if t.startswith("s_waitcnt") and "vmcnt" in t:
                    break
                if t.startswith(".") or (t.startswith("buffer_load_dwordx4") and "offen offset:" in t):
                    continue
                assert not (_regs(t) & dst), f"{name}: `{t}` touches {lines[i]!r} before its wait"
            checked += 1
    assert checked >= 20
