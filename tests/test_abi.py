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


def test_prefill_plans_reject(fa):
    """Instruction-prefill plans, contiguous and paged: host validation before any HIP call."""
    h = _heads(fa)
    out = C.c_void_p()
    create = lambda d: fa.raw_call("fka_plan_create_prefill", C.byref(h), C.byref(d), C.byref(out))
    create_p = lambda d: fa.raw_call("fka_plan_create_prefill_paged", C.byref(h), C.byref(d), C.byref(out))
    assert create(fa.PrefillDesc(5, 0, 100, 64, 64, 0)) == -1 and "n_tokens" in fa.last_error()
    assert create(fa.PrefillDesc(5, 8, 100, 64, 4, 0)) == -1 and "max_suffix_len" in fa.last_error()
    assert create(fa.PrefillDesc(5, 8, 100, 64, 64, -1)) == -1 and "blocks" in fa.last_error()
    assert create(fa.PrefillDesc(64, 9, 100, 64, 64, 0)) == -2  # 576 tokens: more than 512
    #                               N  n  Lp   page max_pages pool msl blocks
    assert create_p(fa.PrefillPagedDesc(5, 8, 100, 8, 64, 100, 32, 0)) == -1 and "page_size" in fa.last_error()
    assert create_p(fa.PrefillPagedDesc(5, 8, 100, 16, 8, 100, 32, 0)) == -1 and "pages" in fa.last_error()
    assert create_p(fa.PrefillPagedDesc(5, 8, 100, 16, 64, 0, 32, 0)) == -1 and "n_pool_pages" in fa.last_error()
    assert create_p(fa.PrefillPagedDesc(5, 8, 100, 16, 64, 100, 4, 0)) == -1 and "max_suffix_len" in fa.last_error()
    assert not out.value
    n = None
    assert fa.raw_call("fka_prefill", n, n, n, n, n, n, n, n, n, n) == -1
    assert fa.raw_call("fka_prefill_paged", n, n, n, n, n, n, n, n, n) == -1


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


def test_misaligned_pointers_are_rejected(fa):
    """Pointers are checked for alignment before anything is launched or dereferenced: 16 bytes for
    bf16 rows and fp32 outputs, 4 for int32 / fp32 arrays.  The addresses here are never read (the
    checks run first), so no GPU is needed."""
    vp = C.c_void_p
    a16, a8, a2 = vp(0x10000), vp(0x10008), vp(0x10002)
    assert fa.raw_call("fka_lse_merge", 4, 2, 64, a8, a16, a16, None, None) == -1
    assert "part_o is not 16-byte aligned" in fa.last_error()
    assert fa.raw_call("fka_lse_merge", 4, 2, 64, a16, a2, a16, None, None) == -1
    assert "part_lse is not 4-byte aligned" in fa.last_error()
    assert fa.raw_call("fka_lse_merge", 4, 2, 64, a16, a16, a8, None, None) == -1
    assert "out is not 16-byte aligned" in fa.last_error()
    assert fa.raw_call("fka_lse_merge", 4, 2, 64, a16, a16, a16, a2, None) == -1
    assert "out_lse is not 4-byte aligned" in fa.last_error()
    assert fa.raw_call("fka_read_probe", a8, C.c_size_t(4096), 1, 64, 4, a16, None) == -1
    assert "buf is not 16-byte aligned" in fa.last_error()
    assert fa.raw_call("fka_scatter_pages", a8, a16, 16, 0, a16, 1, 128, 4, a16, a16, None, None) == -1
    assert "k_src is not 16-byte aligned" in fa.last_error()
    assert fa.raw_call("fka_scatter_pages", a16, a16, 16, 0, a2, 1, 128, 4, a16, a16, None, None) == -1
    assert "page_row is not 4-byte aligned" in fa.last_error()
    h = _heads(fa)
    d = fa.ContigDesc(5, 512, 64, 64, 1, 0, 0)
    good = [a16] * 5 + [a16, a16, None, None]  # q, prefix k/v, suffix k/v, suffix_len, out, out_lse, err
    for i, name, bad in [(0, "q", a8), (1, "prefix_k", a8), (4, "suffix_v", a8), (5, "suffix_len", a2),
                         (6, "out", a8), (7, "out_lse", a2), (8, "err", a2)]:
        args = list(good)
        args[i] = bad
        assert fa.raw_call("fka_fork_decode_noalloc", C.byref(h), C.byref(d), *args, None) == -1, name
        assert f"{name} is not" in fa.last_error(), (name, fa.last_error())


@pytest.mark.gpu
def test_misaligned_pointers_are_rejected_by_plan_calls(fa):
    """The plan entry points refuse views offset from 16-byte (bf16 rows, fp32 outputs) or 4-byte
    (lengths, tables, lse) alignment with FKA_ERR_INVALID_ARG and launch nothing."""
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    plan = fa.Plan.contig(8, 2, 64, 3, 128, 32, 32)
    N, Hq, d = 3, 8, 64
    buf = torch.zeros(1 << 20, dtype=torch.bfloat16, device="cuda")
    i32 = torch.zeros(64, dtype=torch.int32, device="cuda")
    f32 = torch.zeros(1 << 16, dtype=torch.float32, device="cuda")
    vp = C.c_void_p
    b16, b8 = vp(buf.data_ptr()), vp(buf.data_ptr() + 8)
    i4, i2 = vp(i32.data_ptr()), vp(i32.data_ptr() + 2)
    f16, f8, f2 = vp(f32.data_ptr()), vp(f32.data_ptr() + 8), vp(f32.data_ptr() + 2)
    h = plan._h
    good = [b16, b16, b16, b16, b16, i4, f16, f16]  # q, prefix k/v, suffix k/v, suffix_len, out, out_lse
    for i, name, bad in [(0, "q", b8), (2, "prefix_v", b8), (3, "suffix_k", b8), (5, "suffix_len", i2),
                         (6, "out", f8), (7, "out_lse", f2)]:
        args = list(good)
        args[i] = bad
        assert fa.raw_call("fka_fork_decode", h, *args, None) == -1, name
        assert f"{name} is not" in fa.last_error(), (name, fa.last_error())
    assert fa.raw_call("fka_partials", h, b16, b16, b16, b16, b16, i4, f8, f16, None) == -1
    assert "part_o is not 16-byte aligned" in fa.last_error()
    assert fa.raw_call("fka_partials", h, b16, b16, b16, b16, b16, i4, f16, f2, None) == -1
    assert "part_lse is not 4-byte aligned" in fa.last_error()
    torch.cuda.synchronize()
    assert plan.device_error() == 0
