"""The backward recurrence's partial memory-counter waits, checked against the
compiled code (no GPU needed).

In lstm_bwd_xcd each wave copies its k-slice of the exchanged rows in chunks
of direct loads (IPC instructions per chunk), issues its cell inputs as
ordinary loads right after the first chunks, and waits for chunk c with a
partial count: vmcnt(n) lets the last n vector-memory operations stay in
flight.  The counts assume a number of cell-input load instructions; if the
compiler ever emitted fewer (merged loads, say), a wait would let the product
read a chunk that has not landed.  This test compiles the kernels for gfx950
and checks, in every instantiation, that at each chunk wait at least n
vector-memory operations follow the last direct load of the chunk it waits
for.
"""

import os
import re
import shutil
import subprocess

import pytest

from paper_1904_10584_amd import build

SRC = os.path.join(build.CSRC, "lstm_xcd.hip")


def _assembly(tmp_path):
    if not shutil.which(build.HIPCC) and not os.path.exists(build.HIPCC):
        pytest.skip("hipcc not available")
    out = tmp_path / "lstm_xcd.s"
    cmd = [build.HIPCC, *build.FLAGS, "--cuda-device-only", "-S", SRC, "-o", str(out)]
    p = subprocess.run(cmd, capture_output=True, text=True)
    assert p.returncode == 0, p.stderr[-2000:]
    return out.read_text().split("\n")


def _events(lines, start):
    """Vector-memory operations and inline-asm vmcnt waits of the function
    that starts at line `start`, in program text order: ('D',) a direct load
    to LDS, ('M',) any other vector-memory operation, ('W', n) a wait."""
    ev, in_asm = [], False
    for line in lines[start + 1:]:
        s = line.strip()
        if s.startswith(".Lfunc_end"):
            break
        if s.startswith(";;#ASMSTART"):
            in_asm = True
            continue
        if s.startswith(";;#ASMEND"):
            in_asm = False
            continue
        if re.match(r"global_load_lds_", s):
            ev.append(("D",))
        elif re.match(r"(global|buffer|flat)_(load|store|atomic)", s):
            ev.append(("M",))
        elif in_asm and s.startswith("s_waitcnt vmcnt"):
            ev.append(("W", int(re.search(r"vmcnt\((\d+)\)", s).group(1))))
    return ev


def test_backward_chunk_waits_leave_only_later_operations_in_flight(tmp_path):
    lines = _assembly(tmp_path)
    heads = [(i, m) for i, l in enumerate(lines)
             if (m := re.match(r"^(_Z\w*lstm_bwd_xcdILi(\d+)ELi(\d+)ELi(\d+)E\w*):", l))]
    assert heads, "no lstm_bwd_xcd instantiation in the assembly"
    for i, m in heads:
        mt, kw = int(m.group(2)), int(m.group(4))
        ch = 4 if kw >= 4 else kw
        ipc, nch = mt * ch, kw // ch  # direct loads per chunk, chunks per step
        sections = 0
        ops, waits = None, 0
        for e in _events(lines, i):
            if ops is None:
                if e[0] == "D":  # a step's first chunk
                    ops, waits = [e], 0
                continue
            if e[0] != "W":
                ops.append(e)
                continue
            # the wait for chunk `waits`: its last direct load is the
            # ((waits + 1) * ipc)-th of the section
            d = [j for j, o in enumerate(ops) if o[0] == "D"]
            assert len(d) >= (waits + 1) * ipc, (m.group(1), waits, len(d))
            last = d[(waits + 1) * ipc - 1]
            after = len(ops) - last - 1
            assert after >= e[1], (
                f"{m.group(1)}: the wait for chunk {waits} allows {e[1]} operations in "
                f"flight but only {after} follow the chunk")
            waits += 1
            if waits == nch:
                sections += 1
                ops = None
        assert sections >= 1, f"{m.group(1)}: no complete product section found"
