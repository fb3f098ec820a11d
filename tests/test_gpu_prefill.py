"""Instruction prefill (fka_prefill) against the oracle's causal definition.

Branch b appends n instruction tokens over the shared prefix (paper Sec. 3.3): token t's queries
attend to the whole prefix and to b's suffix positions [0, L_b + t].  The reference evaluates that
definition directly: instruction token (b, t) is a sequence of its own over [prefix ; b's suffix up
to L_b + t], computed by the fp64 oracle.  Bar: the gates of tests/gates.py on every row.
"""
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


def _instruction(w, n):
    """The workload's n per-step tokens as each branch's instruction: q [N][n][Hq][d], and the
    suffix buffers with token t's key / value at position L_b + t."""
    N = w.q.shape[0]
    q = np.ascontiguousarray(w.step_q[:n].transpose(1, 0, 2, 3))
    sk, sv = w.suffix_k.copy(), w.suffix_v.copy()
    for b in range(N):
        L = int(w.suffix_len[b])
        sk[b, :, L:L + n] = w.step_k[:n, b].transpose(1, 0, 2)
        sv[b, :, L:L + n] = w.step_v[:n, b].transpose(1, 0, 2)
    return q, sk, sv


def _reference(w, n, q, sk, sv):
    """The causal definition, one oracle sequence per instruction token."""
    N, _, Hq, d = q.shape
    qv = q.reshape(N * n, Hq, d)
    vlen = np.array([int(w.suffix_len[b]) + t + 1 for b in range(N) for t in range(n)], np.int32)
    return oracle.decode_contig(qv, w.prefix_k, w.prefix_v, np.repeat(sk, n, axis=0), np.repeat(sv, n, axis=0),
                                vlen, w.spec.softmax_scale)


def _run(fa, w, n, q, sk, sv, blocks=0, suffix_len=None):
    s = w.spec
    N, _, Hq, d = q.shape
    cap = w.suffix_cap
    plan = fa.Plan.prefill_plan(s.n_q_heads, s.n_kv_heads, s.head_dim, N, n, w.prefix_len, cap, cap, blocks=blocks)
    out = torch.full((N, n, Hq, d), float("nan"), device="cuda")
    lse = torch.full((N, n, Hq), float("nan"), device="cuda")
    ln = dev_i32(w.suffix_len if suffix_len is None else suffix_len)
    plan.prefill(dev_bf16(q), dev_bf16(w.prefix_k), dev_bf16(w.prefix_v), dev_bf16(sk), dev_bf16(sv), ln, out, lse)
    torch.cuda.synchronize()
    return plan, out.cpu().numpy().reshape(N * n, Hq, d), lse.cpu().numpy().reshape(N * n, Hq)


@pytest.mark.parametrize("n", [1, 16, 64])
def test_prefill_long_shape(fa, n):
    """The 32k-prefix agent context (40 query / 8 KV heads, d 128, 5 branches) with n-token
    instructions over existing suffixes of 0..40 tokens; every row of every token checked."""
    w = W.make("long", steps=n, suffix_range=(0, 40), seed=2600 + n)
    q, sk, sv = _instruction(w, n)
    print(f"[prefill] long n={n}: suffix_len {w.suffix_len.tolist()}", flush=True)
    plan, out, lse = _run(fa, w, n, q, sk, sv)
    info = plan.info()
    print(f"[prefill] long n={n}: {info.n_units} units, {info.n_items} items, {info.n_blocks} blocks", flush=True)
    ref, ref_lse = _reference(w, n, q, sk, sv)
    m = gates.assert_gates(out, ref, what=f"prefill long n={n}")
    gates.assert_lse(lse, ref_lse, what=f"prefill long n={n}")
    assert plan.device_error() == 0
    rows_per_head = w.q.shape[0] * n * 5
    if rows_per_head >= 8 * 32:
        _check_tiled_plan(info, n_kv_heads=8, rows_per_head=rows_per_head)
    else:
        # the partial kernel's prefill instantiation: the block sets (units_per_block units of one
        # KV head) are a multiple of the 8 XCDs apart, so that the units of a KV head share its
        # prefix tiles; one round of resident blocks
        P, cus = info.units_per_block, torch.cuda.get_device_properties(0).multi_processor_count
        sets = -(-info.n_units // P) * 8
        assert info.n_blocks % sets == 0 and info.n_blocks <= cus and (P == 1 or info.n_items > cus)
    print(f"[prefill] long n={n} {m}", flush=True)


def _check_tiled_plan(info, n_kv_heads, rows_per_head):
    """Head dim 128 with at least 256 rows per KV head runs the tiled kernel: 32-row units, eight
    per block (one per wave), blocks =
    KV heads x unit groups x prefix ranges in one round of resident blocks, one partial slot per
    range (the KV head varies fastest in the grid, so with 8 KV heads a head's blocks share an XCD)."""
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    assert info.units_per_block == 8 and info.waves_per_block == 8
    assert info.n_units == -(-rows_per_head // 32) and info.n_items == info.n_units * n_kv_heads
    groups = n_kv_heads * -(-info.n_units // 8)
    assert info.n_blocks % groups == 0 and info.n_slots == info.n_blocks // groups
    assert info.n_blocks <= max(cus, groups) and info.rounds == 1


def _random_cases(k, seed):
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(k):
        d = int(rng.choice([64, 128]))
        hkv = int(rng.choice([1, 2, 4, 8]))
        g = int(rng.integers(1, 9))
        nb = int(rng.integers(1, 7))
        n = int(rng.integers(1, 40))
        while nb * n > 512:
            n //= 2
        out.append(dict(head_dim=d, n_kv_heads=hkv, n_q_heads=hkv * g, n_branches=nb, n=n,
                        prefix_len=int(rng.integers(0, 3000)), lo=int(rng.integers(0, 60)),
                        blocks=int(rng.choice([0, 0, 7, 64])), seed=int(rng.integers(1, 1 << 30))))
    return out


@pytest.mark.parametrize("c", _random_cases(10, 2601),
                         ids=lambda c: f"d{c['head_dim']}-kv{c['n_kv_heads']}-q{c['n_q_heads']}-b{c['n_branches']}"
                                       f"-n{c['n']}-p{c['prefix_len']}-blk{c['blocks']}")
def test_prefill_random_shapes(fa, c):
    """Seeded shapes: d 64 / 128, 1..8 KV heads, G 1..8, 1..6 branches, 1..39 tokens, prefixes of
    0..3000 (some not a multiple of the 32-key slice), existing suffixes, explicit grids."""
    _check_case(fa, c)


def test_prefill_harvest_into_the_main_context(fa):
    """Thought harvesting appends the harvested text to the main context (paper Sec. 3.5): one
    sequence (n_branches 1) prefilling n tokens over its snapshot and its own suffix, contiguous
    and paged; every row checked."""
    n = 96
    spec = W.CONFIGS["long"].replace(prefix_len=3000, n_branches=1, suffix_range=(300, 300), steps=n, seed=2740)
    w = W.make(spec)
    q, sk, sv = _instruction(w, n)
    ref, ref_lse = _reference(w, n, q, sk, sv)
    plan, out, lse = _run(fa, w, n, q, sk, sv)
    gates.assert_gates(out, ref, what="harvest contiguous")
    gates.assert_lse(lse, ref_lse, what="harvest contiguous")
    pplan, pout, plse = _run_paged(fa, w, n, q, sk, sv, seed=2741)
    gates.assert_gates(pout, ref, what="harvest paged")
    gates.assert_lse(plse, ref_lse, what="harvest paged")
    assert plan.device_error() == 0 and pplan.device_error() == 0


@pytest.mark.parametrize("g", [32, 40, 64])
def test_prefill_wide_groups(fa, g):
    """d 128 with G = 32 (a 32-row unit is one token) and G = 40 and 64, where a token's rows spread
    over two units (the units do not follow token boundaries)."""
    _check_case(fa, dict(head_dim=128, n_kv_heads=2, n_q_heads=2 * g, n_branches=3, n=3, prefix_len=1000, lo=7,
                         blocks=0, seed=2603 + g))


@pytest.mark.parametrize("case", [dict(hkv=8, g=5, nb=3, n=66), dict(hkv=4, g=5, nb=6, n=70)],
                         ids=["kv8-31units", "kv4-66units"])
def test_prefill_many_units(fa, case):
    """Many 32-row units per KV head, with 8 KV heads (one per XCD) and 4, units straddling
    branches, a last unit group of fewer than eight units and a prefix (700 keys) that is not a
    multiple of the 64-key tile; every row of every token checked, contiguous and paged."""
    n = case["n"]
    spec = W.CONFIGS["long"].replace(prefix_len=700, n_branches=case["nb"], n_kv_heads=case["hkv"],
                                     n_q_heads=case["hkv"] * case["g"], suffix_range=(0, 9), steps=n,
                                     seed=2660 + case["hkv"])
    w = W.make(spec)
    q, sk, sv = _instruction(w, n)
    plan, out, lse = _run(fa, w, n, q, sk, sv)
    info = plan.info()
    print(f"[prefill] many units: {info.n_units} units, {info.n_items} items, {info.n_blocks} blocks", flush=True)
    _check_tiled_plan(info, n_kv_heads=case["hkv"], rows_per_head=case["nb"] * n * case["g"])
    ref, ref_lse = _reference(w, n, q, sk, sv)
    gates.assert_gates(out, ref, what="many units")
    gates.assert_lse(lse, ref_lse, what="many units")
    assert plan.device_error() == 0
    pplan, pout, plse = _run_paged(fa, w, n, q, sk, sv, seed=2670 + case["hkv"])
    _check_tiled_plan(pplan.info(), n_kv_heads=case["hkv"], rows_per_head=case["nb"] * n * case["g"])
    gates.assert_gates(pout, ref, what="many units, paged")
    gates.assert_lse(plse, ref_lse, what="many units, paged")
    assert pplan.device_error() == 0


def _check_case(fa, c):
    spec = W.CONFIGS["mid"].replace(head_dim=c["head_dim"], n_kv_heads=c["n_kv_heads"], n_q_heads=c["n_q_heads"],
                                    n_branches=c["n_branches"], prefix_len=c["prefix_len"],
                                    suffix_range=(c["lo"], c["lo"] + 30), steps=c["n"], seed=c["seed"])
    w = W.make(spec)
    n = c["n"]
    q, sk, sv = _instruction(w, n)
    plan, out, lse = _run(fa, w, n, q, sk, sv, blocks=c["blocks"])
    ref, ref_lse = _reference(w, n, q, sk, sv)
    gates.assert_gates(out, ref, what=str(c))
    gates.assert_lse(lse, ref_lse, what=str(c))
    assert plan.device_error() == 0


@pytest.mark.parametrize("c", [dict(head_dim=128, n_kv_heads=2, n_q_heads=8, n_branches=4, n=20, prefix_len=0, lo=5,
                                      blocks=0, seed=2750),
                                 dict(head_dim=128, n_kv_heads=2, n_q_heads=8, n_branches=4, n=20, prefix_len=1500,
                                      lo=5, blocks=3, seed=2751),
                                 dict(head_dim=128, n_kv_heads=1, n_q_heads=1, n_branches=256, n=2, prefix_len=700,
                                      lo=0, blocks=0, seed=2752),
                                 dict(head_dim=128, n_kv_heads=2, n_q_heads=8, n_branches=4, n=20, prefix_len=40, lo=5,
                                      blocks=0, seed=2753)],
                         ids=["empty-prefix", "one-range", "16-branches-per-unit", "prefix-under-one-tile"])
def test_prefill_tiled_edges(fa, c):
    """The tiled kernel (at least 256 rows per KV head) with no prefix at all (the suffix keys
    only), with an explicit grid of one prefix range, with G = 1 and 2-token instructions of
    256 branches, where a 32-row unit holds 16 branches (each masked to its own suffix), and with a
    prefix shorter than one 64-key tile (no whole tile: every prefix key on the per-wave path)."""
    _check_case(fa, c)


def test_prefill_tiled_nonfinite_instruction_value(fa):
    """A NaN in the value of instruction token 17 of branch 1 (KV head 1) reaches exactly the rows
    that attend to it: branch 1's tokens 17.. on that KV head's query heads.  Its earlier tokens and
    every other branch and KV head stay exact (a row that does not read the key multiplies it by
    p = 0, which must not turn into NaN), contiguous and paged."""
    n, G, hkv = 40, 5, 2
    spec = W.CONFIGS["mid"].replace(n_kv_heads=hkv, n_q_heads=hkv * G, n_branches=3, prefix_len=900,
                                    suffix_range=(3, 30), steps=n, seed=2760)
    w = W.make(spec)
    q, sk, sv = _instruction(w, n)
    ref, _ = _reference(w, n, q, sk, sv)
    bad_b, bad_t, bad_g = 1, 17, 1
    sv[bad_b, bad_g, int(w.suffix_len[bad_b]) + bad_t, 5] = W.BF16_NAN
    N, _, Hq, d = q.shape
    hit = np.zeros((N * n, Hq), bool)
    for t in range(bad_t, n):
        hit[bad_b * n + t, bad_g * G:(bad_g + 1) * G] = True
    plan, out, _ = _run(fa, w, n, q, sk, sv)
    assert plan.info().units_per_block == 8
    pplan, pout, _ = _run_paged(fa, w, n, q, sk, sv, seed=2761)
    for what, o in (("contiguous", out), ("paged", pout)):
        assert np.all(np.isnan(o[hit])), what
        gates.assert_gates(o[~hit], ref[~hit], what=f"rows that do not read the NaN, {what}")
    assert plan.device_error() == 0 and pplan.device_error() == 0


def test_prefill_paired_units_on_the_streaming_path(fa):
    """Fewer than 256 rows per KV head keeps the partial kernel's prefill instantiation; with 64 KV
    heads its items (5 units of 32 rows x 64) outnumber the resident blocks, so an eight-wave block
    takes two units of one KV head, four waves each.  Every row checked, contiguous and paged."""
    n = 30
    spec = W.CONFIGS["long"].replace(prefix_len=700, n_branches=5, n_kv_heads=64, n_q_heads=64,
                                     suffix_range=(0, 9), steps=n, seed=2780)
    w = W.make(spec)
    q, sk, sv = _instruction(w, n)
    plan, out, lse = _run(fa, w, n, q, sk, sv)
    info = plan.info()
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    print(f"[prefill] streaming, paired: {info.n_units} units, {info.n_items} items, {info.n_blocks} blocks",
          flush=True)
    assert info.units_per_block == 2 and info.n_units == 5 and info.n_items > cus
    ref, ref_lse = _reference(w, n, q, sk, sv)
    gates.assert_gates(out, ref, what="paired units, streaming")
    gates.assert_lse(lse, ref_lse, what="paired units, streaming")
    pplan, pout, _ = _run_paged(fa, w, n, q, sk, sv, seed=2781)
    assert pplan.info().units_per_block == 2
    gates.assert_gates(pout, ref, what="paired units, streaming, paged")
    assert plan.device_error() == 0 and pplan.device_error() == 0


def _tiled_case(seed, n=20):
    """A small shape on the tiled kernel: d 128, 2 KV heads x G 4, 4 branches of n tokens
    (320 rows per KV head), a 500-key prefix, suffixes of 10-20 keys."""
    spec = W.CONFIGS["mid"].replace(n_kv_heads=2, n_q_heads=8, n_branches=4, prefix_len=500,
                                    suffix_range=(10, 20), steps=n, seed=seed)
    return W.make(spec), n


def test_prefill_tiled_clamps_and_flags_a_suffix_past_the_bound(fa):
    """The tiled kernel clamps a suffix length above max_suffix_len - n (flag 1); the other
    branches stay exact."""
    w, n = _tiled_case(2790)
    q, sk, sv = _instruction(w, n)
    bad = w.suffix_len.copy()
    bad[1] = w.suffix_cap + 3
    plan, out, lse = _run(fa, w, n, q, sk, sv, suffix_len=bad)
    assert plan.info().units_per_block == 8
    assert plan.device_error() == 1
    ref, ref_lse = _reference(w, n, q, sk, sv)
    rows = [t for t in range(q.shape[0] * n) if t // n != 1]
    gates.assert_gates(out[rows], ref[rows], what="tiled, other branches unaffected")
    gates.assert_lse(lse[rows], ref_lse[rows], what="tiled, other branches unaffected")


@pytest.mark.parametrize("where", ["suffix", "prefix", "prefix-tail"])
def test_prefill_tiled_paged_flags_a_bad_page(fa, where):
    """The tiled kernel over the pool skips a page id outside the pool (its rows read as zeros) and
    raises flag 4: in one branch's suffix row the other branches stay exact; in the shared prefix
    (a page of a whole 64-key tile, or of the last 52 keys past them) the flag is raised."""
    w, n = _tiled_case(2791)
    q, sk, sv = _instruction(w, n)
    s = w.spec
    N, _, Hq, d = q.shape
    kp, vp, table = _to_pool(w, sk, sv, seed=2792)
    npre = -(-w.prefix_len // 16)
    if where == "suffix":
        table[2, npre] = kp.shape[0] + 100
    elif where == "prefix":
        table[:, 3] = kp.shape[0] + 7
    else:
        assert w.prefix_len % 64 == 52
        table[:, npre - 1] = kp.shape[0] + 7
    plan = fa.Plan.prefill_paged_plan(s.n_q_heads, s.n_kv_heads, s.head_dim, N, n, w.prefix_len, table.shape[1],
                                      kp.shape[0], w.suffix_cap)
    assert plan.info().units_per_block == 8
    out = torch.full((N, n, Hq, d), float("nan"), device="cuda")
    plan.prefill_paged(dev_bf16(q), dev_bf16(kp), dev_bf16(vp), dev_i32(table), dev_i32(w.suffix_len), out)
    torch.cuda.synchronize()
    assert plan.device_error() & 4
    o = out.cpu().numpy().reshape(N * n, Hq, d)
    assert np.all(np.isfinite(o))
    if where == "suffix":
        ref, _ = _reference(w, n, q, sk, sv)
        rows = [t for t in range(N * n) if t // n != 2]
        gates.assert_gates(o[rows], ref[rows], what="tiled paged, other branches exact")


def _to_pool(w, sk, sv, seed, spare=5):
    """The prefix and each branch's suffix buffer (instruction tokens included) in a page pool of
    16-token pages whose ids are a seeded permutation: the prefix pages are shared by every
    branch's row, branch b's suffix position u sits at index ceil(Lp / 16) + u // 16."""
    N, Hkv, cap, d = sk.shape
    Lp = w.prefix_len
    npre, nsuf = -(-Lp // 16), -(-cap // 16)
    n_pages = npre + N * nsuf + spare
    perm = np.random.default_rng(seed).permutation(n_pages)
    kp = np.zeros((n_pages, Hkv, 16, d), np.uint16)
    vp = np.zeros_like(kp)
    table = np.full((N, npre + nsuf), -1, np.int32)

    def put(pid, k_src, v_src, lo, hi):
        kp[pid, :, :hi - lo] = k_src[:, lo:hi]
        vp[pid, :, :hi - lo] = v_src[:, lo:hi]

    for i in range(npre):
        put(perm[i], w.prefix_k, w.prefix_v, 16 * i, min(16 * i + 16, Lp))
        table[:, i] = perm[i]
    for b in range(N):
        for j in range(nsuf):
            pid = perm[npre + b * nsuf + j]
            put(pid, sk[b], sv[b], 16 * j, min(16 * j + 16, cap))
            table[b, npre + j] = pid
    return kp, vp, table


def _run_paged(fa, w, n, q, sk, sv, seed, blocks=0):
    s = w.spec
    N, _, Hq, d = q.shape
    kp, vp, table = _to_pool(w, sk, sv, seed)
    plan = fa.Plan.prefill_paged_plan(s.n_q_heads, s.n_kv_heads, s.head_dim, N, n, w.prefix_len, table.shape[1],
                                      kp.shape[0], w.suffix_cap, blocks=blocks)
    out = torch.full((N, n, Hq, d), float("nan"), device="cuda")
    lse = torch.full((N, n, Hq), float("nan"), device="cuda")
    plan.prefill_paged(dev_bf16(q), dev_bf16(kp), dev_bf16(vp), dev_i32(table), dev_i32(w.suffix_len), out, lse)
    torch.cuda.synchronize()
    return plan, out.cpu().numpy().reshape(N * n, Hq, d), lse.cpu().numpy().reshape(N * n, Hq)


@pytest.mark.parametrize("n", [1, 16, 64])
def test_prefill_paged_long_shape(fa, n):
    """The paged prefill at the 32k-prefix shape (40 query / 8 KV heads, d 128, 5 branches): the
    pool's pages in a seeded random order, the prefix pages shared; every row of every token
    against the oracle's causal definition, as for the contiguous layout."""
    w = W.make("long", steps=n, suffix_range=(0, 40), seed=2700 + n)
    q, sk, sv = _instruction(w, n)
    plan, out, lse = _run_paged(fa, w, n, q, sk, sv, seed=2710 + n)
    info = plan.info()
    print(f"[prefill paged] long n={n}: {info.n_units} units, {info.n_blocks} blocks", flush=True)
    ref, ref_lse = _reference(w, n, q, sk, sv)
    m = gates.assert_gates(out, ref, what=f"paged prefill long n={n}")
    gates.assert_lse(lse, ref_lse, what=f"paged prefill long n={n}")
    assert plan.device_error() == 0
    print(f"[prefill paged] long n={n} {m}", flush=True)


@pytest.mark.parametrize("c", _random_cases(6, 2720),
                         ids=lambda c: f"d{c['head_dim']}-kv{c['n_kv_heads']}-q{c['n_q_heads']}-b{c['n_branches']}"
                                       f"-n{c['n']}-p{c['prefix_len']}-blk{c['blocks']}")
def test_prefill_paged_random_shapes(fa, c):
    """Seeded shapes as for the contiguous prefill, over a permuted page pool."""
    spec = W.CONFIGS["mid"].replace(head_dim=c["head_dim"], n_kv_heads=c["n_kv_heads"], n_q_heads=c["n_q_heads"],
                                    n_branches=c["n_branches"], prefix_len=c["prefix_len"],
                                    suffix_range=(c["lo"], c["lo"] + 30), steps=c["n"], seed=c["seed"])
    w = W.make(spec)
    n = c["n"]
    q, sk, sv = _instruction(w, n)
    plan, out, lse = _run_paged(fa, w, n, q, sk, sv, seed=c["seed"] + 1, blocks=c["blocks"])
    ref, ref_lse = _reference(w, n, q, sk, sv)
    gates.assert_gates(out, ref, what="paged " + str(c))
    gates.assert_lse(lse, ref_lse, what="paged " + str(c))
    assert plan.device_error() == 0


def test_prefill_paged_flags_a_bad_page(fa):
    """A page id outside the pool in one branch's suffix row is not read (flag 4); the other
    branches are exact."""
    n = 4
    w = W.make("tiny", steps=n, suffix_range=(10, 20), seed=2730)
    q, sk, sv = _instruction(w, n)
    s = w.spec
    N, _, Hq, d = q.shape
    kp, vp, table = _to_pool(w, sk, sv, seed=2731)
    table[2, -(-w.prefix_len // 16)] = kp.shape[0] + 100
    plan = fa.Plan.prefill_paged_plan(s.n_q_heads, s.n_kv_heads, s.head_dim, N, n, w.prefix_len, table.shape[1],
                                      kp.shape[0], w.suffix_cap)
    out = torch.full((N, n, Hq, d), float("nan"), device="cuda")
    plan.prefill_paged(dev_bf16(q), dev_bf16(kp), dev_bf16(vp), dev_i32(table), dev_i32(w.suffix_len), out)
    torch.cuda.synchronize()
    assert plan.device_error() & 4
    ref, _ = _reference(w, n, q, sk, sv)
    rows = [t for t in range(N * n) if t // n != 2]
    gates.assert_gates(out.cpu().numpy().reshape(N * n, Hq, d)[rows], ref[rows], what="other branches exact")


def test_prefill_clamps_and_flags_a_suffix_past_the_bound(fa):
    """A suffix length above max_suffix_len - n is clamped to it (and flagged), like a decode's."""
    n = 5
    w = W.make("tiny", steps=n, suffix_range=(10, 20), seed=2602)
    q, sk, sv = _instruction(w, n)
    cap = w.suffix_cap
    bad = w.suffix_len.copy()
    bad[1] = cap + 3
    plan, out, lse = _run(fa, w, n, q, sk, sv, suffix_len=bad)
    assert plan.device_error() == 1
    # branch 1 now reads up to its clamped bound (the NaN past its data); the others are exact
    ref, ref_lse = _reference(w, n, q, sk, sv)
    N = q.shape[0]
    rows = [s for s in range(N * n) if s // n != 1]
    gates.assert_gates(out[rows], ref[rows], what="other branches unaffected")
    gates.assert_lse(lse[rows], ref_lse[rows], what="other branches unaffected")


def test_prefill_plan_rejects_other_calls(fa):
    """A prefill plan serves fka_prefill only; decode entry points refuse it."""
    plan = fa.Plan.prefill_plan(8, 2, 64, 3, 4, 100, 32, 32)
    t = torch.zeros(1 << 16, dtype=torch.bfloat16, device="cuda")
    ln = torch.zeros(3, dtype=torch.int32, device="cuda")
    o = torch.zeros(1 << 14, dtype=torch.float32, device="cuda")
    with pytest.raises(fa.FkaError, match="prefill"):
        plan.decode(t, t, t, t, t, ln, o)
    tab = torch.zeros((3, 16), dtype=torch.int32, device="cuda")
    with pytest.raises(fa.FkaError, match="paged"):
        plan.prefill_paged(t, t, t, tab, ln, o)
    pp = fa.Plan.prefill_paged_plan(8, 2, 64, 3, 4, 100, 16, 64, 32)
    with pytest.raises(fa.FkaError, match="paged"):
        pp.prefill(t, t, t, t, t, ln, o)
    with pytest.raises(fa.FkaError, match="prefill"):
        pp.decode_paged(t, t, t, tab, ln, o)
