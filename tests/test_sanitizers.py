"""The host-side C/C++ under AddressSanitizer + UndefinedBehaviorSanitizer (tests/sanitize.sh): the
oracle with its pins, the library's host code (page pool, plan validation, ABI checks) with the pool,
ABI and schedule tests, and the schedule arithmetic checker.  CPU only; about a minute."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.slow
def test_host_code_is_clean_under_asan_and_ubsan():
    if not (shutil.which("gcc") and os.path.exists("/opt/rocm/bin/hipcc")):
        pytest.skip("gcc or hipcc missing")
    r = subprocess.run(["bash", os.path.join(ROOT, "tests", "sanitize.sh")], capture_output=True, text=True,
                       timeout=900)
    assert r.returncode == 0 and "[sanitize] clean" in r.stdout, (r.stdout[-4000:] + r.stderr[-4000:])
