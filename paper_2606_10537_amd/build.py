"""Build the HIP library ``libpd.so`` for gfx950 with hipcc (in-tree).

Usage: ``python -m paper_2606_10537_amd.build`` or ``build()`` from Python.
"""

import concurrent.futures
import os
import subprocess
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
INCLUDE = os.path.join(ROOT, "include")
BUILD = os.path.join(PKG, "_build")
LIB = os.path.join(PKG, "libpd.so")
SOURCES = ["pd_api.hip", "attn_bf16.hip", "attn_f32.hip", "select.hip", "diag.hip"]
ARCH = "gfx950"

HIPCC = os.environ.get("HIPCC", "/opt/rocm/bin/hipcc")
FLAGS = [
    f"--offload-arch={ARCH}", "-O3", "-std=c++17", "-fPIC",
    "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops",
    "-Wno-unused-result", f"-I{INCLUDE}", f"-I{CSRC}",
]


# Per-source extra flags.  The bf16 attention kernels never create or test NaN
# (masked scores are -inf), so NaN semantics are dropped there: the row maxima
# then compile to v_max3_f32 chains without canonicalising each MFMA output.
EXTRA = {"attn_bf16.hip": ["-fno-honor-nans"]}


def _run(cmd):
    r = subprocess.run(cmd, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, text=True)
    out = "\n".join(l for l in r.stdout.splitlines() if "packed-fp32-ops" not in l)
    if r.returncode != 0:
        raise RuntimeError(f"command failed ({r.returncode}): {' '.join(cmd)}\n{out}")
    return out


# The checking build: kernels verify every kept chunk and slot index (see
# pd_common.h); the library the path loads is the release build.
LIB_CHECK = os.path.join(PKG, "libpd_check.so")


def build(verbose: bool = False) -> str:
    """Compile every source for gfx950 and link libpd.so and the index-checking libpd_check.so; returns
    the path of libpd.so."""
    variants = [(LIB, BUILD, []), (LIB_CHECK, os.path.join(BUILD, "check"), ["-DPD_CHECK_INDICES=1"])]
    cmds, links = [], []
    for lib, objdir, defines in variants:
        os.makedirs(objdir, exist_ok=True)
        objs = [os.path.join(objdir, s.replace(".hip", ".o")) for s in SOURCES]
        cmds += [[HIPCC, *FLAGS, *defines, *EXTRA.get(s, []), "-c", os.path.join(CSRC, s), "-o", o]
                 for s, o in zip(SOURCES, objs)]
        links.append((lib, objs))
    with concurrent.futures.ThreadPoolExecutor(max_workers=8) as ex:
        for out in ex.map(_run, cmds):
            if verbose and out.strip():
                print(out)
    for lib, objs in links:
        tmp = lib + ".tmp"
        _run([HIPCC, f"--offload-arch={ARCH}", "-shared", "-fPIC", *objs, "-o", tmp])
        os.replace(tmp, lib)
    return LIB


if __name__ == "__main__":
    print(build(verbose="-v" in sys.argv))
