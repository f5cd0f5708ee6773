"""The C ABI's host-side validation built with AddressSanitizer and UndefinedBehaviorSanitizer (host
code only: the sanitizer flags sit after -Xarch_host, so no GPU code is built with them) and driven by
tests/sanitize/abi_driver.cpp, which calls every entry point with arguments it must reject before
anything is launched.  Runs on the CPU: a rejected call never reaches the HIP runtime."""

import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2606_10537_amd")
OUT = os.path.join(PKG, "_build", "sanitize")
HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")


def run(cmd, **kw):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True, **kw)
    return r.returncode, r.stdout


@pytest.mark.skipif(not os.path.exists(HIPCC), reason="hipcc not installed")
def test_abi_validation_under_asan_ubsan():
    sys.path.insert(0, ROOT)
    from paper_2606_10537_amd import build as B
    os.makedirs(OUT, exist_ok=True)
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer", "-g"]
    objs = []
    for src in B.SOURCES:
        o = os.path.join(OUT, src.replace(".hip", ".o"))
        extra = san if src == "pd_api.hip" else []
        rc, out = run([B.HIPCC, *B.FLAGS, *B.EXTRA.get(src, []), *extra, "-c", os.path.join(B.CSRC, src), "-o", o])
        assert rc == 0, out[-3000:]
        objs.append(o)
    drv = os.path.join(OUT, "abi_driver.o")
    rc, out = run([B.HIPCC, "-x", "c++", "-std=c++17", "-O1", *san, f"-I{B.INCLUDE}", "-c",
                   os.path.join(ROOT, "tests", "sanitize", "abi_driver.cpp"), "-o", drv])
    assert rc == 0, out[-3000:]
    exe = os.path.join(OUT, "abi_driver")
    rc, out = run([B.HIPCC, f"--offload-arch={B.ARCH}", *san, drv, *objs, "-o", exe])
    assert rc == 0, out[-3000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1", HIP_VISIBLE_DEVICES="")
    rc, out = run([exe], env=env, timeout=120)
    assert rc == 0 and "ok (0 failures)" in out, out[-4000:]
    assert "ERROR: AddressSanitizer" not in out and "runtime error" not in out, out[-4000:]
