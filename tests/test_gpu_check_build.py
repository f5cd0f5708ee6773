"""The index-checking build (libpd_check.so, compiled with PD_CHECK_INDICES): out-of-range kept chunks
or slots turn the outputs that depend on them into NaN, with every access still in bounds, while valid
indices give the release results.  Runs tests/check_build_probe.py in a fresh process (one library per
process)."""

import json
import os
import subprocess
import sys

import pytest

pytestmark = pytest.mark.gpu
HERE = os.path.dirname(os.path.abspath(__file__))


def test_checking_build_flags_out_of_range_indices():
    print("[check build] probe: decode (bf16, fp32, splits 1 and 3), gather, joint gather", flush=True)
    r = subprocess.run([sys.executable, os.path.join(HERE, "check_build_probe.py")], capture_output=True, text=True,
                       timeout=300)
    lines = [l for l in r.stdout.splitlines() if l.startswith("{")]
    assert lines, r.stdout[-2000:] + r.stderr[-3000:]
    checks = json.loads(lines[-1])
    failed = [k for k, v in checks.items() if not v]
    assert r.returncode == 0 and not failed, failed
