"""The gradient kernel streams its operands into LDS with direct-to-LDS copies
(global_load_lds) and waits for them with partial `s_waitcnt vmcnt(N)`.
Copies complete in issue order among themselves, but an ordinary vector
memory operation issued after a copy may complete before it; vmcnt counts
both, so a partial wait reached while such an operation is in flight can
pass before the copy it waits for has landed.  The kernel therefore issues
no ordinary load or store between its copies and their partial waits.

This checks that rule on the built gfx950 code objects: over the control
flow graph of every gradient kernel (loops iterated to a fixpoint), no
partial vmcnt wait is reachable from an ordinary vector memory operation
that was issued after a copy with no `vmcnt(0)` in between."""
import os
import re
import shutil
import subprocess
import tempfile

import pytest

from paper_2412_06464_amd import gdn

OBJDUMP = "/opt/rocm/llvm/bin/llvm-objdump"
FUNC = re.compile(r"^([0-9a-f]+) <(\S+)>:$")
INS = re.compile(r"^\s+([a-z_0-9]+)\b(.*?)//\s*([0-9A-F]+):")
TARGET = re.compile(r"<(\S+)\+0x([0-9a-f]+)>")
ORDINARY = re.compile(r"^(global|buffer|flat|scratch)_(load|store|atomic)")
VMCNT = re.compile(r"vmcnt\((\d+)\)")


def functions(text):
    """{name: [(address, opcode, operands, branch target or None)]}"""
    out, cur, base = {}, None, 0
    for ln in text.splitlines():
        m = FUNC.match(ln)
        if m:
            base, cur = int(m.group(1), 16), m.group(2)
            out[cur] = []
            continue
        m = INS.match(ln)
        if m and cur:
            t = TARGET.search(ln)
            tgt = None
            if m.group(1).startswith(("s_branch", "s_cbranch")) and t and t.group(1) == cur:
                tgt = base + int(t.group(2), 16)
            out[cur].append((int(m.group(3), 16), m.group(1), m.group(2), tgt))
    return out


def violations(ins):
    """Partial vmcnt waits reachable with an ordinary memory operation issued
    after a copy still possibly in flight.  State per program point: (a copy
    issued since the last vmcnt(0), an ordinary operation issued after it);
    a point is re-walked whenever the state arriving there grows (the
    transfer is gen/kill per flag, so this reaches the fixpoint)."""
    index = {a: i for i, (a, _, _, _) in enumerate(ins)}
    seen = {}
    work, bad = [(0, (False, False))], set()
    while work:
        i, (dma, after) = work.pop()
        while i is not None:
            old = seen.get(i, (False, False))
            state = (dma or old[0], after or old[1])
            if i in seen and state == old:
                break  # nothing new arrives here
            seen[i] = state
            dma, after = state
            _, op, args, tgt = ins[i]
            if op.startswith("global_load_lds") or (op.startswith("buffer_load") and " lds" in args):
                dma = True
            elif ORDINARY.match(op):
                after = after or dma
            elif op == "s_waitcnt":
                m = VMCNT.search(args)
                if m and int(m.group(1)) == 0:
                    dma = after = False
                elif m and int(m.group(1)) < 63 and after:
                    bad.add(ins[i][0])
            if op == "s_endpgm" or op.startswith("s_setpc"):
                break
            if tgt is not None:
                work.append((index[tgt], (dma, after)))
            i = i + 1 if not op.startswith("s_branch") and i + 1 < len(ins) else None
    return sorted(bad)


@pytest.mark.skipif(not os.path.exists(OBJDUMP), reason="llvm-objdump not available")
def test_partial_waits_never_follow_ordinary_memory_ops_after_copies():
    if not os.path.exists(gdn.LIB_PATH):
        from paper_2412_06464_amd import build
        build.build()
    tmp = tempfile.mkdtemp()
    try:
        lib = os.path.join(tmp, "libgdn.so")
        shutil.copy(gdn.LIB_PATH, lib)
        subprocess.run([OBJDUMP, "--offloading", lib], cwd=tmp, check=True, capture_output=True)
        objs = [os.path.join(tmp, f) for f in os.listdir(tmp) if f.endswith("gfx950")]
        assert objs, "no gfx950 code object in libgdn.so"
        checked = 0
        for obj in objs:
            text = subprocess.run([OBJDUMP, "-d", "--mcpu=gfx950", obj], check=True,
                                  capture_output=True, text=True).stdout
            for name, ins in functions(text).items():
                if "6k_grad" not in name or not ins:
                    continue
                assert any(op.startswith("global_load_lds") for _, op, _, _ in ins), name
                assert violations(ins) == [], (name, [hex(a) for a in violations(ins)])
                checked += 1
        assert checked >= 4  # the gradient kernels of every supported shape
    finally:
        shutil.rmtree(tmp)


def test_checker_flags_a_planted_early_wait():
    """The checker itself: an ordinary load issued between a copy and its
    partial wait is flagged (in a loop, on the second trip round); with a
    vmcnt(0) in between, or the load before the copy, it is not."""
    def prog(lines):
        return [(4 * i, op, args, tgt) for i, (op, args, tgt) in enumerate(lines)]
    looped = prog([("s_waitcnt", " vmcnt(2)", None),        # 0: loop head
                   ("global_load_lds_dwordx4", " v1, s[0:1]", None),
                   ("global_load_dwordx4", " v[2:5], v1, s[0:1]", None),
                   ("s_cbranch_scc1", " -4", 0),               # back to the head
                   ("s_endpgm", "", None)])
    assert violations(looped) == [0]
    fixed = prog([("s_waitcnt", " vmcnt(2)", None),
                  ("global_load_lds_dwordx4", " v1, s[0:1]", None),
                  ("s_waitcnt", " vmcnt(0)", None),
                  ("global_load_dwordx4", " v[2:5], v1, s[0:1]", None),
                  ("s_cbranch_scc1", " -5", 0),
                  ("s_endpgm", "", None)])
    assert violations(fixed) == []
    before = prog([("global_load_dwordx4", " v[2:5], v1, s[0:1]", None),
                   ("global_load_lds_dwordx4", " v1, s[0:1]", None),
                   ("s_waitcnt", " vmcnt(1)", None),
                   ("s_endpgm", "", None)])
    assert violations(before) == []
