"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

Two drivers in tests/sanitize/ are built with -fsanitize=address,undefined
(the HIP sources with the sanitizers on their host side only) and run with
leak detection and abort-on-error:
  * oracle_driver.c runs the fp64 oracle (oracle/gdn_oracle.c, built here
    with gcc) on dense and packed problems with empty and one-token
    sequences, with and without states, several checkpoint spacings;
  * api_driver.c runs libgdn's host side (gdn_api.hip, gdn_launch.hip:
    argument checks, packed-boundary validation, workspace sizing, the
    pointer audit) linked against the kernel objects of the regular build;
    none of its calls reaches a HIP call.
"""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = os.path.join(ROOT, "tests", "sanitize")
CSRC = os.path.join(ROOT, "paper_2412_06464_amd", "csrc")
KBUILD = os.path.join(ROOT, "paper_2412_06464_amd", "_build")
ENV = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1",
           UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
HOST_SAN = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
            "-Xarch_host", "-fno-sanitize-recover=undefined", "-Xarch_host",
            "-fno-omit-frame-pointer"]


def run(cmd, **kw):
    r = subprocess.run(cmd, capture_output=True, text=True, **kw)
    assert r.returncode == 0, "%s\n%s%s" % (" ".join(cmd), r.stdout, r.stderr[-4000:])
    return r


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_oracle_under_asan_ubsan(tmp_path):
    exe = str(tmp_path / "oracle_driver")
    run(["gcc", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
         "-fno-omit-frame-pointer", os.path.join(ROOT, "oracle", "gdn_oracle.c"),
         os.path.join(SAN, "oracle_driver.c"), "-lm", "-lpthread", "-o", exe])
    r = run([exe], env=ENV, timeout=300)
    assert "oracle driver: ok" in r.stdout


def _kernel_objects():
    """Objects of the kernel translation units from the regular build
    (built here if absent)."""
    names = ("gdn_prep", "gdn_seq", "gdn_grad", "gdn_recurrent", "gdn_block")
    objs = [os.path.join(KBUILD, n + ".o") for n in names]
    if not all(os.path.exists(o) for o in objs):
        from paper_2412_06464_amd import build
        build.build()
    return objs


@pytest.mark.skipif(not os.path.exists("/opt/rocm/bin/hipcc"), reason="needs hipcc")
def test_host_library_under_asan_ubsan(tmp_path):
    from paper_2412_06464_amd.build import FLAGS, HIPCC
    objs = []
    for n in ("gdn_api", "gdn_launch"):
        o = str(tmp_path / (n + ".o"))
        flags = [f for f in FLAGS if f != "-O3"] + ["-O1", "-g"]
        run([HIPCC, *flags, *HOST_SAN, "-c", os.path.join(CSRC, n + ".hip"), "-o", o])
        objs.append(o)
    clang = "/opt/rocm/llvm/bin/clang"
    drv = str(tmp_path / "api_driver.o")
    run([clang, "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
         "-c", os.path.join(SAN, "api_driver.c"), "-o", drv])
    exe = str(tmp_path / "api_driver")
    run([clang + "++", "-fsanitize=address,undefined", drv, *objs, *_kernel_objects(),
         "-L/opt/rocm/lib", "-lamdhip64", "-Wl,-rpath,/opt/rocm/lib", "-o", exe])
    r = run([exe], env=ENV, timeout=300)
    assert "api driver: ok" in r.stdout
