"""Static check of the kernels' hand-issued LDS reads (CPU only: needs hipcc).

The decode loops of attn_partial_kernel and attn_token_kernel issue their
table, pair and query reads in inline assembly and wait for them with their
own `s_waitcnt lgkmcnt(N)`, so that the key and value chains overlap.  The
compiler sees neither the reads nor what they are waiting for: correctness
rests on two facts about the code it emits, checked here on the gfx950
device assembly of every instantiation, built with the library's own flags:

* no instruction reads or writes the destination registers of such a read
  (a register copy, a spill, reuse for another value) before a wait covers
  it;
* a wait with count N covers a read when at least N LDS operations were
  issued after it (LDS operations of a wavefront complete in order; scalar
  loads, which also count, only make a wait stricter), and no branch or
  label lies between a read and its wait.
"""

import os
import re
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

REG_RANGE = re.compile(r"\b([vas])\[(\d+):(\d+)\]")
REG_ONE = re.compile(r"\b([vas])(\d+)\b")
BRANCH = ("s_cbranch", "s_branch", "s_setpc", "s_endpgm")


def _regs(text):
    out = set()
    for k, a, b in REG_RANGE.findall(text):
        out.update((k, i) for i in range(int(a), int(b) + 1))
    for k, a in REG_ONE.findall(REG_RANGE.sub(" ", text)):
        out.add((k, int(a)))
    return out


def _lgkm_limit(ops):
    m = re.search(r"lgkmcnt\((\d+)\)", ops)
    if m:
        return int(m.group(1))
    return 0 if ops.strip() == "0" else None


def _functions(text):
    name, body = None, []
    for line in text.split("\n"):
        m = re.match(r"\s*\.type\s+([^,]+),@function", line)
        if m:
            if name:
                yield name, body
            name, body = m.group(1), []
        elif name:
            if line.startswith(".Lfunc_end"):
                yield name, body
                name, body = None, []
            else:
                body.append(line)
    if name:
        yield name, body


def check_function(body):
    """(problems, number of inline-asm LDS reads) for one function's lines."""
    problems, pending = [], []     # pending: (destination registers, LDS index)
    in_asm, nlds, nreads = False, 0, 0
    for no, line in enumerate(body):
        s = line.strip()
        if s == ";;#ASMSTART":
            in_asm = True
            continue
        if s == ";;#ASMEND":
            in_asm = False
            continue
        if not line[:1].isspace() and s.split(";")[0].strip().endswith(":"):   # a label: control may arrive from elsewhere
            if pending:
                problems.append((no, "label while asm reads are pending", s))
                pending = []
            continue
        if not s or s.startswith(";") or s.startswith("."):
            continue
        s = s.split(";")[0].strip()
        mn, _, ops = s.partition(" ")
        if mn == "s_waitcnt":
            n = _lgkm_limit(ops)
            if n is not None:
                pending = [p for p in pending if nlds - 1 - p[1] < n]
            continue
        touched = _regs(ops)
        for dest, _ in pending:
            if dest & touched:
                problems.append((no, "touches a pending destination", s))
        if mn.startswith(BRANCH) and pending:
            problems.append((no, "branch while asm reads are pending", s))
            pending = []
        if mn.startswith("ds_"):
            if in_asm and mn.startswith(("ds_read", "ds_load")):
                pending.append((_regs(ops.split(",")[0]), nlds))
                nreads += 1
            nlds += 1
    return problems, nreads


def _fn(lines):
    return [l if l.split(";")[0].strip().endswith(":") else "\t" + l for l in lines]


def test_checker_catches_planted_mistakes():
    read = [";;#ASMSTART", "ds_read_b64 v[2:3], v1 offset:8", ";;#ASMEND"]
    use = ["v_add_u32_e32 v4, v2, v5"]
    ok = lambda lines: check_function(_fn(lines))[0] == []
    assert ok(read + [";;#ASMSTART", "s_waitcnt lgkmcnt(0)", ";;#ASMEND"] + use)
    # one LDS operation issued after the read: lgkmcnt(1) covers it
    assert ok(read + ["ds_write_b32 v7, v8", ";;#ASMSTART", "s_waitcnt lgkmcnt(1)", ";;#ASMEND"] + use)
    # no wait, a wait that does not cover it, a wait on vmcnt only
    assert not ok(read + use)
    assert not ok(read + ["s_waitcnt lgkmcnt(1)"] + use)
    assert not ok(read + ["s_waitcnt vmcnt(0)"] + use)
    # a copy, an overwrite, the high half of the pair, a branch, a label
    assert not ok(read + ["v_mov_b32 v9, v3"])
    assert not ok(read + ["v_mov_b32 v2, 0"])
    assert not ok(read + ["v_mfma_i32_4x4x4_16b_i8 a[0:3], v9, v[2:3], a[0:3]"])
    assert not ok(read + ["s_cbranch_scc1 .LBB0_2", "s_waitcnt lgkmcnt(0)"])
    assert not ok(read + [".LBB0_2:", "s_waitcnt lgkmcnt(0)"])
    assert not ok(read + [".LBB0_3:                                ; =>This Inner Loop Header: Depth=1",
                          "s_waitcnt lgkmcnt(0)"])
    # registers elsewhere are free to use
    assert ok(read + ["v_mov_b32 v9, v4", "s_waitcnt lgkmcnt(0)"] + use)


@pytest.mark.timeout(600)
def test_inline_lds_reads_are_waited_for(tmp_path):
    import __graft_entry__ as ge

    if not os.path.exists(ge.HIPCC) and shutil.which("hipcc") is None:
        pytest.skip("hipcc not available")
    flags = [f for f in ge.FLAGS if f not in ("-shared", "-fPIC")]
    procs = {}
    for src in ("dq_decode.hip", "dq_token.hip"):
        out = str(tmp_path / (src + ".s"))
        cmd = [ge.HIPCC, *flags, "--cuda-device-only", "-S", os.path.join(ge.CSRC, src), "-o", out]
        procs[src] = (subprocess.Popen(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT), out)
    reads = {}
    for src, (p, out) in procs.items():
        log = p.communicate()[0]
        assert p.returncode == 0, log.decode(errors="replace")[-2000:]
        for name, body in _functions(open(out).read()):
            problems, n = check_function(body)
            assert problems == [], (name, problems[:5])
            reads[name] = n
    partial = [n for k, n in reads.items() if "attn_partial_kernel" in k]
    token = [n for k, n in reads.items() if "attn_token_kernel" in k]
    assert partial and token
    # every entropy-coded instantiation decodes through the hand-issued reads
    # (the fixed-width one does not decode)
    assert sum(n > 0 for n in partial) >= len(partial) - 1
    assert all(n > 0 for n in token)
