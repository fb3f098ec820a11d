"""Host logic of the work schedule (no GPU): the arithmetic shared by the partial kernel,
the merge kernel and fka_plan_slots, checked for coverage and slot invariants on
random item sizes and grids by tests/native/sched_check.cpp."""
import os
import shutil
import subprocess
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _hipcc():
    for c in (os.environ.get("HIPCC"), "/opt/rocm/bin/hipcc", shutil.which("hipcc")):
        if c and os.path.exists(c):
            return c
    pytest.skip("hipcc not found")


def test_schedule_invariants():
    with tempfile.TemporaryDirectory() as d:
        exe = os.path.join(d, "sched_check")
        subprocess.run([_hipcc(), "-std=c++17", "-O2", "-I", os.path.join(ROOT, "paper_2608_13667_amd", "csrc"),
                        os.path.join(ROOT, "tests", "native", "sched_check.cpp"), "-o", exe],
                       check=True, capture_output=True, cwd=d)
        r = subprocess.run([exe, "3000"], capture_output=True, text=True, timeout=120)
        assert r.returncode == 0 and r.stdout.startswith("ok"), r.stdout + r.stderr
