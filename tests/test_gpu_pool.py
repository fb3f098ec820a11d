"""The K/V lifecycle of a fork on the device, through the C ABI: the snapshot scattered into pool
pages, five sequences forked off it (fka_pool_fork), decode steps with appends into pages the pool
reserves ahead, harvest (the four branches dropped), the main sequence promoted to the next
snapshot (fka_pool_promote, a gather of the tail, fka_scatter_pages) and a second turn forked off that.  Outputs
are checked against the oracle over the materialised contexts; the gathers bit-exactly."""
import math

import numpy as np
import pytest
import torch

import oracle
from paper_2608_13667_amd import workloads as W
from tests import gates
from tests.gpu_util import dev_bf16, dev_i32

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def fa():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_13667_amd import forkattn
    return forkattn


def _bf16(rng, shape):
    return W.bf16_bits(rng.standard_normal(shape, dtype=np.float32))


def test_fork_lifecycle_on_device(fa):
    Hq, Hkv, d, N = 16, 4, 128, 5
    Lp, S1, S2 = 1000, 37, 21  # 1000 = 62 pages + 8 tokens: the last prefix page is shared, partly filled
    n_pages, max_pages = 160, 72
    scale = 1.0 / math.sqrt(d)
    rng = np.random.default_rng(2608)
    prefix_k, prefix_v = _bf16(rng, (Hkv, Lp, d)), _bf16(rng, (Hkv, Lp, d))
    pool = fa.Pool(n_pages)
    k_pool = dev_bf16(np.full((n_pages, Hkv, 16, d), W.BF16_NAN, np.uint16))
    v_pool = dev_bf16(np.full((n_pages, Hkv, 16, d), W.BF16_NAN, np.uint16))
    err = torch.zeros(1, dtype=torch.int32, device="cuda")

    def turn(plan, table, lp, ctx_k, ctx_v, steps, what):
        """steps fused append + decode steps on all N sequences, pages reserved one token ahead."""
        suf_k = np.full((N, Hkv, steps, d), W.BF16_NAN, np.uint16)
        suf_v = np.full((N, Hkv, steps, d), W.BF16_NAN, np.uint16)
        lens = dev_i32(np.zeros(N, np.int32))
        out = torch.empty((N, Hq, d), device="cuda")
        lse = torch.empty((N, Hq), device="cuda")
        for t in range(steps):
            for b in range(N):
                pool.reserve(table, b, lp, t + 1)
            q, kn, vn = _bf16(rng, (N, Hq, d)), _bf16(rng, (N, Hkv, d)), _bf16(rng, (N, Hkv, d))
            suf_k[:, :, t], suf_v[:, :, t] = kn, vn
            plan.step_paged(dev_bf16(q), dev_bf16(kn), dev_bf16(vn), k_pool, v_pool, dev_i32(table), lens, out, lse)
            if t in (0, steps - 1):
                torch.cuda.synchronize()
                ref, ref_lse = oracle.decode_contig(q, ctx_k, ctx_v, suf_k, suf_v, np.full(N, t + 1, np.int32), scale)
                print(f"[pool] {what} step {t}", flush=True)
                gates.assert_gates(out.cpu().numpy(), ref, what=f"{what} step {t}")
                gates.assert_lse(lse.cpu().numpy(), ref_lse, what=f"{what} step {t}")
        assert lens.cpu().tolist() == [steps] * N
        return suf_k, suf_v

    # turn 1: the snapshot into pages, five sequences forked off it
    snap = pool.alloc(-(-Lp // 16))
    fa.scatter_pages(dev_bf16(prefix_k), dev_bf16(prefix_v), 0, dev_i32(snap), n_pages, k_pool, v_pool, err)
    table = np.full((N, max_pages), -1, np.int32)
    pool.fork(snap, table, 0, N)
    pool.release(snap)
    assert pool.refcount(int(snap[-1])) == N
    plan1 = fa.Plan.paged_plan(Hq, Hkv, d, [0, N], [Lp], max_pages, n_pages, S1)
    suf_k, suf_v = turn(plan1, table, Lp, prefix_k, prefix_v, S1, "turn 1")

    # harvest: the branches end; the main sequence's context becomes the next snapshot
    for b in range(1, N):
        pool.drop(table, b)
    assert pool.refcount(int(snap[-1])) == 1
    L0 = Lp + S1
    ctx_k = np.concatenate([prefix_k, suf_k[0]], axis=1)
    ctx_v = np.concatenate([prefix_v, suf_v[0]], axis=1)
    old_table = dev_i32(table)
    dense, frm = pool.promote(table, 0, Lp, S1)
    assert frm == (Lp // 16) * 16 and len(dense) == -(-L0 // 16)
    tmp_k = torch.empty((Hkv, L0 - frm, d), dtype=torch.bfloat16, device="cuda")
    tmp_v = torch.empty_like(tmp_k)
    plan1.gather_paged_range(0, frm, L0, k_pool, v_pool, old_table, tmp_k, tmp_v)  # before the scatter
    fa.scatter_pages(tmp_k, tmp_v, frm, dev_i32(dense), n_pages, k_pool, v_pool, err)
    torch.cuda.synchronize()
    assert np.array_equal(tmp_k.cpu().view(torch.int16).numpy().view(np.uint16), ctx_k[:, frm:])
    assert np.array_equal(tmp_v.cpu().view(torch.int16).numpy().view(np.uint16), ctx_v[:, frm:])

    # turn 2: five sequences forked off the promoted context
    table2 = np.full((N, max_pages), -1, np.int32)
    pool.fork(dense, table2, 0, N)
    pool.release(dense)
    plan2 = fa.Plan.paged_plan(Hq, Hkv, d, [0, N], [L0], max_pages, n_pages, S2)
    g_k = torch.empty((Hkv, L0, d), dtype=torch.bfloat16, device="cuda")
    g_v = torch.empty_like(g_k)
    plan2.gather_paged(3, k_pool, v_pool, dev_i32(table2), L0, g_k, g_v)
    torch.cuda.synchronize()
    assert np.array_equal(g_k.cpu().view(torch.int16).numpy().view(np.uint16), ctx_k)
    assert np.array_equal(g_v.cpu().view(torch.int16).numpy().view(np.uint16), ctx_v)
    turn(plan2, table2, L0, ctx_k, ctx_v, S2, "turn 2")

    for b in range(N):
        pool.drop(table2, b)
    assert pool.free_pages() == n_pages
    assert int(err.item()) == 0
    assert plan1.device_error() == 0 and plan2.device_error() == 0


def test_branch_instruction_prefill(fa):
    """Each branch appends a short instruction (n tokens, causal among themselves) over the shared
    prefix (Sec. 3.3: the snapshot followed by a branch-specific instruction), on the page pool
    after a fork: once as one paged decode over N*n virtual sequences in one group -- token t of
    branch b is a sequence whose page row is b's and whose suffix length is L_b + t + 1 -- and once
    through fka_prefill_paged on the same pages.  Both are checked against the oracle's causal
    definition: query (b, t) attends to the prefix and to b's suffix positions [0, L_b + t]."""
    Hq, Hkv, d, N, n = 16, 4, 128, 5, 3  # 5 * 3 virtual sequences x 4 q heads = 60 rows per KV head
    Lp, n_pages, max_pages = 1000, 120, 70
    scale = 1.0 / math.sqrt(d)
    rng = np.random.default_rng(4242)
    Lb = rng.integers(0, 41, size=N)
    prefix_k, prefix_v = _bf16(rng, (Hkv, Lp, d)), _bf16(rng, (Hkv, Lp, d))
    cap = int(Lb.max()) + n
    suf_k = np.full((N, Hkv, cap, d), W.BF16_NAN, np.uint16)
    suf_v = np.full((N, Hkv, cap, d), W.BF16_NAN, np.uint16)
    for b in range(N):
        suf_k[b, :, :Lb[b] + n] = _bf16(rng, (Hkv, Lb[b] + n, d))
        suf_v[b, :, :Lb[b] + n] = _bf16(rng, (Hkv, Lb[b] + n, d))
    pool = fa.Pool(n_pages)
    k_pool = dev_bf16(np.full((n_pages, Hkv, 16, d), W.BF16_NAN, np.uint16))
    v_pool = dev_bf16(np.full((n_pages, Hkv, 16, d), W.BF16_NAN, np.uint16))
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    snap = pool.alloc(-(-Lp // 16))
    fa.scatter_pages(dev_bf16(prefix_k), dev_bf16(prefix_v), 0, dev_i32(snap), n_pages, k_pool, v_pool, err)
    table = np.full((N, max_pages), -1, np.int32)
    pool.fork(snap, table, 0, N)
    pool.release(snap)
    a = -(-Lp // 16)
    for b in range(N):  # the branch's suffix so far and its instruction, through the suffix layout
        pool.reserve(table, b, Lp, int(Lb[b]) + n)
        fa.scatter_pages(dev_bf16(suf_k[b, :, :Lb[b] + n]), dev_bf16(suf_v[b, :, :Lb[b] + n]), 0,
                         dev_i32(table[b, a:]), n_pages, k_pool, v_pool, err)
    vt = np.repeat(table, n, axis=0)                                      # row b*n + t is branch b's
    vlen = np.array([Lb[b] + t + 1 for b in range(N) for t in range(n)], np.int32)
    q = _bf16(rng, (N * n, Hq, d))
    plan = fa.Plan.paged_plan(Hq, Hkv, d, [0, N * n], [Lp], max_pages, n_pages, int(vlen.max()))
    out = torch.empty((N * n, Hq, d), device="cuda")
    lse = torch.empty((N * n, Hq), device="cuda")
    plan.decode_paged(dev_bf16(q), k_pool, v_pool, dev_i32(vt), dev_i32(vlen), out, lse)
    torch.cuda.synchronize()
    ref, ref_lse = oracle.decode_contig(q, prefix_k, prefix_v, np.repeat(suf_k, n, axis=0),
                                        np.repeat(suf_v, n, axis=0), vlen, scale)
    gates.assert_gates(out.cpu().numpy(), ref, what="instruction prefill")
    gates.assert_lse(lse.cpu().numpy(), ref_lse, what="instruction prefill")
    assert int(err.item()) == 0 and plan.device_error() == 0
    info = plan.info()
    # one item per KV head holding all N * n * G rows: the prefix is read once per chunk
    assert info.n_units == 1 and info.n_items == Hkv and info.slot_rows == N * n * (Hq // Hkv)
    # the same instruction through the prefill kernel on the same pool and page rows
    pplan = fa.Plan.prefill_paged_plan(Hq, Hkv, d, N, n, Lp, max_pages, n_pages, cap)
    out2 = torch.empty((N, n, Hq, d), device="cuda")
    lse2 = torch.empty((N, n, Hq), device="cuda")
    pplan.prefill_paged(dev_bf16(q.reshape(N, n, Hq, d)), k_pool, v_pool, dev_i32(table), dev_i32(Lb), out2, lse2)
    torch.cuda.synchronize()
    gates.assert_gates(out2.cpu().numpy().reshape(N * n, Hq, d), ref, what="paged prefill kernel")
    gates.assert_lse(lse2.cpu().numpy().reshape(N * n, Hq), ref_lse, what="paged prefill kernel")
    assert pplan.device_error() == 0


def test_ranged_gather_bit_exact(fa):
    """fka_gather_paged_range copies exactly logical positions [begin, end) of a sequence, across
    the prefix / suffix boundary, the partly filled prefix page and empty ranges."""
    w = W.make(W.CONFIGS["paged"].replace(n_tasks=3, prefix_range=(1, 400), suffix_range=(0, 90), n_kv_heads=2,
                                          n_q_heads=8, seed=94))
    from tests.gpu_util import paged_plan, to_dev_paged
    plan = paged_plan(fa, w)
    dv = to_dev_paged(w)
    rng = np.random.default_rng(95)
    for i in range(w.n_seqs):
        t = i // w.spec.n_branches
        Lp, Ls = int(w.prefix_len[t]), int(w.suffix_len[i])
        rk, rv = oracle.gather_paged(w.k_pool, w.v_pool, w.page_table, i, Lp, Ls)
        for begin, end in ((0, Lp + Ls), (Lp, Lp + Ls), (max(Lp - 5, 0), min(Lp + 7, Lp + Ls)),
                           tuple(sorted(rng.integers(0, Lp + Ls + 1, size=2))), (Lp + Ls, Lp + Ls)):
            begin, end = int(begin), int(end)
            ko = torch.full((w.spec.n_kv_heads, max(end - begin, 1), w.spec.head_dim), 7.0, dtype=torch.bfloat16,
                            device="cuda")
            vo = torch.full_like(ko, 7.0)
            plan.gather_paged_range(i, begin, end, dv["k_pool"], dv["v_pool"], dv["page_table"], ko, vo)
            torch.cuda.synchronize()
            n = end - begin
            assert np.array_equal(ko.view(torch.int16).cpu().numpy().view(np.uint16)[:, :n], rk[:, begin:end])
            assert np.array_equal(vo.view(torch.int16).cpu().numpy().view(np.uint16)[:, :n], rv[:, begin:end])
    assert plan.device_error() == 0


def test_scatter_skips_and_flags_bad_page_ids(fa):
    """A page id outside the pool is not written: its positions are skipped, bit 4 is raised in the
    error word, and the valid pages still receive their positions."""
    Hkv, d, n_pages = 2, 64, 6
    rng = np.random.default_rng(96)
    src_k, src_v = _bf16(rng, (Hkv, 40, d)), _bf16(rng, (Hkv, 40, d))
    k_pool = dev_bf16(np.full((n_pages, Hkv, 16, d), W.BF16_NAN, np.uint16))
    v_pool = dev_bf16(np.full((n_pages, Hkv, 16, d), W.BF16_NAN, np.uint16))
    err = torch.zeros(1, dtype=torch.int32, device="cuda")
    row = np.array([4, n_pages + 3, 1], np.int32)  # positions 16..31 have no valid page
    fa.scatter_pages(dev_bf16(src_k), dev_bf16(src_v), 0, dev_i32(row), n_pages, k_pool, v_pool, err)
    torch.cuda.synchronize()
    assert int(err.item()) == 4
    kp = k_pool.view(torch.int16).cpu().numpy().view(np.uint16)
    assert np.array_equal(kp[4], src_k[:, 0:16])
    assert np.array_equal(kp[1, :, :8], src_k[:, 32:40])
    assert np.all(kp[1, :, 8:] == W.BF16_NAN) and np.all(kp[[0, 2, 3, 5]] == W.BF16_NAN)
