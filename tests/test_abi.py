"""The C-ABI library: it loads, exports every function include/forkattn.h declares,
and rejects bad arguments on the host with the documented status codes (no GPU needed:
validation happens before any HIP call)."""
import ctypes as C
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def fa():
    from paper_2608_13667_amd import forkattn
    return forkattn


def _declared():
    src = open(os.path.join(ROOT, "include", "forkattn.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(fka_[a-z_]+)\s*\(", src)))


def test_header_declares_the_boundary():
    names = _declared()
    for must in ("fka_fork_decode", "fka_fork_decode_paged", "fka_partials", "fka_lse_merge", "fka_gather_paged",
                 "fka_append_kv", "fka_plan_create_contig", "fka_plan_create_paged"):
        assert must in names


def test_library_exports_every_declared_symbol(fa):
    lib = C.CDLL(fa.LIB_PATH)
    for name in _declared():
        assert hasattr(lib, name), name
    assert set(_declared()) == set(fa.EXPORTED)


def test_version_and_empty_error(fa):
    assert fa.version() == 20000
    assert isinstance(fa.last_error(), str)


def _heads(fa, hq=8, hkv=2, d=64, scale=0.0):
    return fa.Heads(hq, hkv, d, scale)


def _create(fa, heads, desc):
    out = C.c_void_p()
    st = fa.raw_call("fka_plan_create_contig", C.byref(heads) if heads is not None else None,
                     C.byref(desc) if desc is not None else None, C.byref(out))
    return st, out


@pytest.mark.parametrize("heads,desc,status,needle", [
    (None, (5, 512, 64, 64, 1, 0), -1, "heads is null"),
    ((8, 3, 64), (5, 512, 64, 64, 1, 0), -1, "multiple"),
    ((8, 2, 96), (5, 512, 64, 64, 1, 0), -2, "head_dim"),
    ((8, 2, 64), (0, 512, 64, 64, 1, 0), -1, "n_branches"),
    ((8, 2, 64), (5, -1, 64, 64, 1, 0), -1, "prefix_len"),
    ((8, 2, 64), (5, 512, 64, 65, 1, 0), -1, "max_suffix_len"),
    ((8, 2, 64), (5, 512, 0, 0, 1, 0), -1, "suffix_cap"),
    ((8, 2, 64), (5, 512, 64, 64, 2, 0), -1, "share_prefix"),
    ((8, 2, 64), (5, 512, 64, 64, 1, 100), -1, "rounds"),
    ((8, 2, 64), (5, 512, 64, 64, 1, -1), -1, "rounds"),
    ((8, 8, 64), (513, 512, 64, 64, 0, 0), -2, "sequences"),
    ((128, 2, 64), (2, 512, 64, 64, 1, 0), -2, "rows"),
    ((64, 8, 128), (9, 512, 64, 64, 1, 0), -2, "rows"),
    # suffixes whose slices would overflow the schedule's 32-bit arithmetic
    ((8, 2, 64), (512, 512, 2**31 - 1, 2**31 - 1, 0, 0), -2, "too long"),
    ((8, 2, 64), (512, 512, 2**25, 2**25, 0, 0), -2, "too long"),
    ((8, 2, 64), (5, 2**31 - 1, 64, 64, 1, 0), -2, "too long"),
])
def test_plan_create_rejects(fa, heads, desc, status, needle):
    h = _heads(fa, *heads) if heads else None
    d = fa.ContigDesc(*desc)
    st, out = _create(fa, h, d)
    assert st == status
    assert needle in fa.last_error()
    assert not out.value


def test_plan_create_rejects_bad_scale(fa):
    st, _ = _create(fa, _heads(fa, scale=float("nan")), fa.ContigDesc(5, 512, 64, 64, 1, 0))
    assert st == -1 and "softmax_scale" in fa.last_error()


def test_paged_plan_rejects(fa):
    import numpy as np
    h = _heads(fa)
    gs = np.array([0, 5], np.int32)
    gl = np.array([100], np.int32)
    out = C.c_void_p()
    vp = lambda a: a.ctypes.data_as(C.c_void_p)
    d = fa.PagedDesc(5, 1, 8, 64, 100, 32, 1, 0)        # page size 8
    assert fa.raw_call("fka_plan_create_paged", C.byref(h), C.byref(d), vp(gs), vp(gl), C.byref(out)) == -1
    d = fa.PagedDesc(5, 1, 16, 4, 100, 32, 1, 0)        # table too narrow for 100 + 32 tokens
    assert fa.raw_call("fka_plan_create_paged", C.byref(h), C.byref(d), vp(gs), vp(gl), C.byref(out)) == -1
    assert "pages" in fa.last_error()
    gs2 = np.array([0, 0, 5], np.int32)
    gl2 = np.array([10, 10], np.int32)
    d = fa.PagedDesc(5, 2, 16, 64, 100, 32, 1, 0)       # empty group
    assert fa.raw_call("fka_plan_create_paged", C.byref(h), C.byref(d), vp(gs2), vp(gl2), C.byref(out)) == -1
    assert "empty" in fa.last_error()


def test_calls_with_null_plan_are_rejected(fa):
    n = None
    assert fa.raw_call("fka_fork_decode", n, n, n, n, n, n, n, n, n, n) == -1
    assert fa.raw_call("fka_fork_decode_paged", n, n, n, n, n, n, n, n, n) == -1
    assert fa.raw_call("fka_append_kv", n, n, n, n, n, n, n) == -1
    assert fa.raw_call("fka_gather_paged", n, 0, n, n, n, 0, n, n, n) == -1
    assert fa.raw_call("fka_gather_paged_range", n, 0, 0, 0, n, n, n, n, n, n) == -1
    assert fa.raw_call("fka_scatter_pages", n, n, 4, 5, n, 1, 128, 1, n, n, n, n) == -1  # from > len
    assert fa.raw_call("fka_plan_get_info", n, n) == -1
    assert fa.raw_call("fka_plan_slots", n, n, n, 0, n) == -1
    fa.raw_call("fka_plan_destroy", n)   # NULL is ignored


def test_lse_merge_rejects_head_dim(fa):
    assert fa.raw_call("fka_lse_merge", 4, 2, 96, None, None, None, None, None) == -2
    assert fa.raw_call("fka_lse_merge", -1, 2, 64, None, None, None, None, None) == -1
    assert fa.raw_call("fka_lse_merge", 0, 2, 64, None, None, None, None, None) == 0


def test_binding_rejects_host_and_mistyped_tensors(fa):
    """The binding hands the library device pointers only: a host tensor, a wrong dtype or a
    non-contiguous view is refused before any call (an int64 length array would otherwise be
    read as int32 pairs, a host pointer would reach the kernels)."""
    import torch
    with pytest.raises(ValueError, match="GPU"):
        fa._p(torch.zeros(4, dtype=torch.int32), "i32")
    with pytest.raises(ValueError):
        fa._p(torch.zeros(4).numpy(), "f32")
    assert fa._p(None, "f32") is None


def test_plan_create_rejects_negative_blocks(fa):
    st, out = _create(fa, _heads(fa), fa.ContigDesc(5, 512, 64, 64, 1, 0, -1))
    assert st == -1 and "blocks" in fa.last_error() and not out.value
