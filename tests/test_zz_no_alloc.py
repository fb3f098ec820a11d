"""The no-allocation decode (fka_fork_decode_noalloc, on the library's static scratch) against the
plan decode (fka_fork_decode) it is a variant of: the same schedule for the same sizes, so the same
outputs bit for bit, on two calls in a row (the second smaller, so it runs over what the first
left in the scratch), plus the oracle's gates, the error word and the size limit."""
import ctypes as C

import numpy as np
import pytest
import torch

import oracle
from paper_2608_13667_amd import workloads as W
from tests import gates
from tests.gpu_util import contig_plan, dev_i32, run_contig, to_dev_contig

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def fa():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_13667_amd import forkattn
    return forkattn


def _noalloc(fa, w, dv, err=None, rounds=0, blocks=0):
    s = w.spec
    N, Hq, d = dv["q"].shape
    out = torch.full((N, Hq, d), float("nan"), device="cuda")
    lse = torch.full((N, Hq), float("nan"), device="cuda")
    fa.decode_noalloc(s.n_q_heads, s.n_kv_heads, s.head_dim, w.prefix_len, w.suffix_cap, w.suffix_cap, dv["q"],
                      dv["prefix_k"], dv["prefix_v"], dv["suffix_k"], dv["suffix_v"], dv["suffix_len"], out, lse,
                      err=err, rounds=rounds, blocks=blocks)
    torch.cuda.synchronize()
    return out.cpu().numpy(), lse.cpu().numpy()


def test_noalloc_matches_plan_decode_on_two_calls(fa):
    """A mid-shaped decode, then a smaller one (fewer heads, shorter prefix, another head_dim):
    each equals the plan decode bit for bit and passes the oracle's gates."""
    cases = [W.make("mid", prefix_len=5000, steps=0, seed=71), W.make("tiny", prefix_len=900, steps=0, seed=72)]
    for i, w in enumerate(cases):
        print(f"[noalloc] call {i}: {w.spec.name} q {w.q.shape} prefix {w.prefix_len}", flush=True)
        dv = to_dev_contig(w)
        err = torch.zeros(1, dtype=torch.int32, device="cuda")
        out, lse = _noalloc(fa, w, dv, err=err)
        plan = contig_plan(fa, w)
        ref_out, ref_lse = run_contig(plan, dv, w.spec.n_q_heads)
        assert np.array_equal(out, ref_out), f"call {i}: output differs from the plan decode"
        assert np.array_equal(lse, ref_lse), f"call {i}: lse differs from the plan decode"
        o_ref, l_ref = oracle.decode_workload(w)
        gates.assert_gates(out, o_ref, what=f"noalloc call {i}")
        gates.assert_lse(lse, l_ref, what=f"noalloc call {i}")
        assert int(err.item()) == 0 and plan.device_error() == 0


def test_noalloc_explicit_grid_and_clamp_flag(fa):
    """An explicit grid (rounds and blocks as a plan would take them) and a suffix length past
    the bound: the call clamps it like the plan decode and sets flag 1 in the caller's word."""
    w = W.make("mid", prefix_len=2000, steps=0, seed=73)
    dv = to_dev_contig(w)
    ln = w.suffix_len.copy()
    ln[2] = w.suffix_cap + 7
    dv["suffix_len"] = dev_i32(ln)
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    out, lse = _noalloc(fa, w, dv, err=err, rounds=3, blocks=40)
    plan = contig_plan(fa, w, rounds=3, blocks=40)
    ref_out, ref_lse = run_contig(plan, dv, w.spec.n_q_heads)
    # the clamped sequence reads positions past its generated suffix, which hold NaN: both NaN
    assert np.isnan(out[2]).all() and np.array_equal(out, ref_out, equal_nan=True)
    assert np.array_equal(lse, ref_lse, equal_nan=True)
    assert int(err.item()) == 1
    assert plan.device_error() == 1


def test_noalloc_rejects_what_it_cannot_hold(fa):
    """More partial results than the scratch holds, or a naive (unshared) schedule: a clear error,
    nothing launched."""
    w = W.make("mid", prefix_len=2000, steps=0, seed=74)
    dv = to_dev_contig(w)
    with pytest.raises(fa.FkaError, match="scratch"):
        _noalloc(fa, w, dv, rounds=64)
    s = w.spec
    h = fa.Heads(s.n_q_heads, s.n_kv_heads, s.head_dim, 0.0)
    d = fa.ContigDesc(w.n_branches, w.prefix_len, w.suffix_cap, w.suffix_cap, 0, 0, 0)
    out = torch.empty((w.n_branches, s.n_q_heads, s.head_dim), device="cuda")
    st = fa.raw_call("fka_fork_decode_noalloc", C.byref(h), C.byref(d), C.c_void_p(dv["q"].data_ptr()),
                     C.c_void_p(dv["prefix_k"].data_ptr()), C.c_void_p(dv["prefix_v"].data_ptr()),
                     C.c_void_p(dv["suffix_k"].data_ptr()), C.c_void_p(dv["suffix_v"].data_ptr()),
                     C.c_void_p(dv["suffix_len"].data_ptr()), C.c_void_p(out.data_ptr()), None, None, None)
    assert st != 0 and "share_prefix" in fa.last_error()
