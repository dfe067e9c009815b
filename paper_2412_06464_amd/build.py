"""Build libgdn.so (HIP, gfx950) in-tree with hipcc.

    python -m paper_2412_06464_amd.build
"""
from __future__ import annotations

import concurrent.futures as cf
import os
import subprocess
import sys

HERE = os.path.dirname(os.path.abspath(__file__))
CSRC = os.path.join(HERE, "csrc")
LIB = os.path.join(HERE, "libgdn.so")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
ARCH = "gfx950"
SOURCES = ["gdn_prep.hip", "gdn_seq.hip", "gdn_grad.hip", "gdn_recurrent.hip", "gdn_block.hip",
           "gdn_launch.hip", "gdn_api.hip"]
FLAGS = ["--offload-arch=" + ARCH, "-O3", "-std=c++20", "-fPIC",
         # keep the compiler from emitting packed fp32 math
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]


def _compile(src: str, obj: str, extra=()) -> None:
    cmd = [HIPCC, *FLAGS, *extra, "-c", os.path.join(CSRC, src), "-o", obj]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("hipcc failed for %s:\n%s%s" % (src, r.stdout, r.stderr))


def build(verbose: bool = False, out: str = LIB, defines=()) -> str:
    """Compile every source for gfx950 and link ``out``.  ``defines`` are
    extra -D flags (tuning experiments; the defaults are the product)."""
    extra = ["-D" + d for d in defines]
    tag = "_".join(d.replace("=", "") for d in defines)
    bdir = os.path.join(HERE, "_build" + ("_" + tag if tag else ""))
    os.makedirs(bdir, exist_ok=True)
    objs = [os.path.join(bdir, os.path.splitext(s)[0] + ".o") for s in SOURCES]
    with cf.ThreadPoolExecutor(len(SOURCES)) as ex:
        list(ex.map(lambda a: _compile(*a, extra), zip(SOURCES, objs)))
    LIBOUT = out
    tmp = LIBOUT + ".tmp%d" % os.getpid()
    cmd = [HIPCC, "--offload-arch=" + ARCH, "-shared", "-fPIC", *objs, "-o", tmp]
    r = subprocess.run(cmd, capture_output=True, text=True)
    if r.returncode != 0:
        raise RuntimeError("link failed:\n%s%s" % (r.stdout, r.stderr))
    os.replace(tmp, LIBOUT)
    if verbose:
        print("built", LIBOUT)
    return LIBOUT


if __name__ == "__main__":
    import argparse
    ap = argparse.ArgumentParser()
    ap.add_argument("--out", default=LIB)
    ap.add_argument("-D", dest="defines", action="append", default=[])
    args = ap.parse_args()
    build(verbose=True, out=os.path.abspath(args.out), defines=args.defines)
    sys.exit(0)
