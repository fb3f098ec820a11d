"""Every read of a matrix-core result in the partial kernel and the tiled prefill kernel is at least
tests.xdl_hazards.MIN_WAIT wait states after the op, in every instantiation of this build (CPU:
compiles the kernels to AMD assembly).  Guards the padding the q.k score reads need beyond the
toolchain's own."""
import os
import shutil
import tempfile

import pytest

from tests import xdl_hazards as X

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.mark.slow
def test_every_xdl_result_read_is_padded():
    hipcc = next((c for c in ("/opt/rocm/bin/hipcc", shutil.which("hipcc")) if c and os.path.exists(c)), None)
    if hipcc is None:
        pytest.skip("hipcc not found")
    with tempfile.TemporaryDirectory() as d:
        asm = X.compile_asm(hipcc, os.path.join(ROOT, "paper_2608_13667_amd", "csrc", "partials.hip"),
                            os.path.join(ROOT, "include"), os.path.join(d, "partials.s"))
    ks = X.kernels(asm)
    assert len(ks) >= 16
    worst = []
    for k in ks:
        pairs = X.scan(asm, k)
        assert pairs, k
        worst.append((min(p[0] for p in pairs), k))
    assert min(worst)[0] >= X.MIN_WAIT, sorted(worst)[:3]


@pytest.mark.slow
def test_every_xdl_result_read_is_padded_in_the_prefill_kernel():
    hipcc = next((c for c in ("/opt/rocm/bin/hipcc", shutil.which("hipcc")) if c and os.path.exists(c)), None)
    if hipcc is None:
        pytest.skip("hipcc not found")
    with tempfile.TemporaryDirectory() as d:
        asm = X.compile_asm(hipcc, os.path.join(ROOT, "paper_2608_13667_amd", "csrc", "prefill.hip"),
                            os.path.join(ROOT, "include"), os.path.join(d, "prefill.s"))
    ks = X.kernels(asm, "prefill_tiles_kernel")
    assert len(ks) == 2
    for k in ks:
        pairs = X.scan(asm, k)
        assert pairs, k
        assert min(p[0] for p in pairs) >= X.MIN_WAIT, (k, sorted(pairs)[:3])
