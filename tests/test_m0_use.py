"""The LDS-DMA statements of the state passes and the gradient kernel set
m0 (the LDS address of a global_load_lds copy) from inline assembly.  The
compiler reserves m0 and does not honour it as a clobber, so the kernels
rely on the compiler never keeping a value of its own in m0.  This checks
the built gfx950 code objects: every instruction that names m0 is a write
of m0 that is directly followed by an LDS-DMA copy, and no instruction that
reads m0 implicitly (relative addressing, messages, GWS) appears."""
import os
import re
import shutil
import subprocess
import tempfile

import pytest

from paper_2412_06464_amd import gdn

OBJDUMP = "/opt/rocm/llvm/bin/llvm-objdump"
IMPLICIT_M0 = re.compile(r"^(s_movrel|v_movrel|s_sendmsg|ds_gws|v_interp|lds_param|ds_.*addtid)")


@pytest.mark.skipif(not os.path.exists(OBJDUMP), reason="llvm-objdump not available")
def test_m0_written_only_by_lds_dma_statements():
    if not os.path.exists(gdn.LIB_PATH):
        from paper_2412_06464_amd import build
        build.build()
    tmp = tempfile.mkdtemp()
    try:
        lib = os.path.join(tmp, "libgdn.so")
        shutil.copy(gdn.LIB_PATH, lib)
        subprocess.run([OBJDUMP, "--offloading", lib], cwd=tmp, check=True,
                       capture_output=True)
        objs = [os.path.join(tmp, f) for f in os.listdir(tmp) if f.endswith("gfx950")]
        assert objs, "no gfx950 code object in libgdn.so"
        dma_copies = 0
        for obj in objs:
            text = subprocess.run([OBJDUMP, "-d", "--mcpu=gfx950", obj], check=True,
                                  capture_output=True, text=True).stdout
            ins = [ln.split("//")[0].strip() for ln in text.splitlines()]
            ins = [x for x in ins if x and re.match(r"^[a-z_0-9]+", x) and not x.endswith(">:")]
            for i, x in enumerate(ins):
                op = x.split()[0]
                assert not IMPLICIT_M0.match(op), (obj, x)
                if re.search(r"\bm0\b", x):
                    assert op == "s_mov_b32" and x.split()[1].rstrip(",") == "m0", (obj, x)
                    nxt = ins[i + 1].split()[0]
                    assert nxt.startswith("global_load_lds"), (obj, x, ins[i + 1])
                    dma_copies += 1
                elif op.startswith("global_load_lds"):
                    prev = ins[i - 1]
                    assert prev.startswith("s_mov_b32") and re.search(r"\bm0\b", prev), (obj, x)
        assert dma_copies > 0
    finally:
        shutil.rmtree(tmp)
