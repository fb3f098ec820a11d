"""GPU parity: the HIP path through the C ABI against the fp64 oracle on the same seeded inputs.

Bar (tests/gates.py): max-abs error <= 2e-3 and max-rel error (floored at the output
RMS) <= 1e-2 on the attention output; |lse error| <= 2e-3; bit-exact for gathers.
All five workloads run at their full sizes with every output row checked.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2608_13667_amd import workloads as W
from tests import gates
from tests.gpu_util import (contig_plan, dev_bf16, dev_i32, paged_plan, run_contig, run_paged, to_dev_contig,
                            to_dev_paged)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def fa():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2608_13667_amd import forkattn
    return forkattn


def _check_contig(fa, w, **plan_kw):
    ref, ref_lse = oracle.decode_workload(w)
    plan = contig_plan(fa, w, **plan_kw)
    out, lse = run_contig(plan, to_dev_contig(w), w.spec.n_q_heads)
    m = gates.assert_gates(out, ref, what=w.spec.name)
    gates.assert_lse(lse, ref_lse, what=w.spec.name)
    assert plan.device_error() == 0
    return m


@pytest.mark.parametrize("name", ["tiny", "tiny-unscaled", "mid", "long", "very-long", "onset"])
def test_config_parity(fa, name):
    spec = W.CONFIGS[name].replace(steps=0)
    print(f"[parity] {name}", flush=True)
    m = _check_contig(fa, W.make(spec))
    print(f"[parity] {name} {m}", flush=True)


def test_paged_config_parity(fa):
    w = W.make("paged")
    print("[parity] paged", flush=True)
    ref, ref_lse = oracle.decode_workload(w)
    plan = paged_plan(fa, w)
    out, lse = run_paged(plan, to_dev_paged(w))
    m = gates.assert_gates(out, ref, what="paged")
    gates.assert_lse(lse, ref_lse, what="paged")
    assert plan.device_error() == 0
    print(f"[parity] paged {m}", flush=True)


def test_long_decode_loop_with_appends(fa):
    """Long agent context: 256 steps, each appending one token per branch then attending."""
    w = W.make("long")
    s = w.spec
    plan = contig_plan(fa, w)
    dv = to_dev_contig(w)
    N, Hq, d = w.q.shape
    out = torch.empty((N, Hq, d), device="cuda")
    lse = torch.empty((N, Hq), device="cuda")
    kn, vn, qn = dev_bf16(w.step_k), dev_bf16(w.step_v), dev_bf16(w.step_q)
    check = {0, 1, 127, 255}
    for t in range(s.steps):
        plan.step(qn[t], kn[t], vn[t], dv["prefix_k"], dv["prefix_v"], dv["suffix_k"], dv["suffix_v"],
                  dv["suffix_len"], out, lse)
        # host mirror of the append for the oracle
        for b in range(N):
            L = int(w.suffix_len[b])
            w.suffix_k[b, :, L] = w.step_k[t, b]
            w.suffix_v[b, :, L] = w.step_v[t, b]
            w.suffix_len[b] = L + 1
        if t in check:
            torch.cuda.synchronize()
            ref, ref_lse = oracle.decode_contig(w.step_q[t], w.prefix_k, w.prefix_v, w.suffix_k, w.suffix_v,
                                                w.suffix_len, s.softmax_scale)
            print(f"[parity] long step {t}", flush=True)
            gates.assert_gates(out.cpu().numpy(), ref, what=f"long step {t}")
            gates.assert_lse(lse.cpu().numpy(), ref_lse, what=f"long step {t}")
    assert np.array_equal(dv["suffix_len"].cpu().numpy(), w.suffix_len)
    # the device suffix buffers hold exactly the appended rows
    L0 = w.suffix_len - s.steps
    for b in range(N):
        got = dv["suffix_k"][b, :, L0[b]:w.suffix_len[b]].view(torch.int16).cpu().numpy().view(np.uint16)
        assert np.array_equal(got, w.suffix_k[b, :, L0[b]:w.suffix_len[b]])
    assert plan.device_error() == 0


@pytest.mark.parametrize("name", ["mid", "tiny-unscaled"])
def test_naive_per_branch_baseline(fa, name):
    _check_contig(fa, W.make(name), share_prefix=False)


@pytest.mark.parametrize("case", [
    dict(prefix_len=0),                                   # no shared prefix at all
    dict(suffix_range=(0, 0)),                            # every suffix empty
    dict(prefix_len=1000),                                # prefix not a multiple of the tile
    dict(prefix_len=1, suffix_range=(0, 3)),              # one prefix token
    dict(n_branches=1),                                   # a single sequence (plain decode)
    dict(n_branches=8, n_q_heads=64, n_kv_heads=8),       # 64 rows per KV head (4 row tiles)
    dict(n_branches=3, n_q_heads=48, n_kv_heads=8),       # 18 rows (2 row tiles, ragged)
    dict(n_q_heads=8, n_kv_heads=8),                      # G = 1 (multi-head attention)
    dict(n_q_heads=24, n_kv_heads=8, n_branches=2),       # 6 rows per KV head
])
def test_edge_cases(fa, case):
    spec = W.CONFIGS["mid"].replace(prefix_len=2048, suffix_range=(0, 300), seed=77).replace(**case)
    print(f"[edge] {case}", flush=True)
    _check_contig(fa, W.make(spec))


def _random_shapes(n, seed):
    """Seeded random plan shapes within the plan limits: GQA group, branches, head_dim, prefix and
    suffix lengths (ragged, some empty), rounds and sharing."""
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(n):
        d = int(rng.choice([64, 128]))
        hkv = int(rng.choice([1, 2, 4, 8]))
        g = int(rng.integers(1, 17))
        nb = int(rng.integers(1, 9))
        while nb * g > 64:  # at most 64 query rows per KV head
            nb -= 1
        lo = int(rng.integers(0, 400))
        out.append(dict(head_dim=d, n_kv_heads=hkv, n_q_heads=hkv * g, n_branches=nb,
                        prefix_len=int(rng.integers(0, 4000)), suffix_range=(lo, lo + int(rng.integers(0, 400))),
                        seed=int(rng.integers(1, 1 << 30)), share=bool(rng.integers(0, 4) > 0),
                        rounds=int(rng.choice([0, 0, 0, 2, 7]))))
    return out


@pytest.mark.parametrize("case", _random_shapes(16, 2026), ids=lambda c: "d{head_dim}-kv{n_kv_heads}-q{n_q_heads}-b{n_branches}-"
                         "p{prefix_len}-s{suffix_range[0]}_{suffix_range[1]}-r{rounds}-{share}".format(**c))
def test_random_shapes(fa, case):
    """Parity on seeded random shapes (not tied to a named workload)."""
    c = dict(case)
    share, rounds = c.pop("share"), c.pop("rounds")
    spec = W.CONFIGS["mid"].replace(**c)
    print(f"[random] {case}", flush=True)
    _check_contig(fa, W.make(spec), share_prefix=share, rounds=rounds)


@pytest.mark.parametrize("rounds", [1, 3, 64])
def test_explicit_rounds(fa, rounds):
    """More rounds: the keys spread over more, smaller partials (64 rounds: ~1 slice per wave)."""
    spec = W.CONFIGS["mid"].replace(prefix_len=3000, seed=78)
    _check_contig(fa, W.make(spec), rounds=rounds)


def test_head_dim_64_full_rows(fa):
    spec = W.CONFIGS["tiny-unscaled"].replace(prefix_len=5000, suffix_range=(100, 700), seed=79)
    _check_contig(fa, W.make(spec))


def test_all_sequences_empty(fa):
    spec = W.CONFIGS["tiny"].replace(prefix_len=0, suffix_range=(0, 0))
    w = W.make(spec)
    plan = contig_plan(fa, w)
    out, lse = run_contig(plan, to_dev_contig(w), spec.n_q_heads)
    assert np.array_equal(out, np.zeros_like(out)) and np.all(np.isneginf(lse))


def test_identical_queries_empty_suffixes_identical_outputs(fa):
    w = W.make("mid", suffix_range=(0, 0))
    w.q[:] = w.q[0:1]
    out, lse = run_contig(contig_plan(fa, w), to_dev_contig(w), 32)
    for b in range(1, w.n_branches):
        assert np.array_equal(out[b], out[0]) and np.array_equal(lse[b], lse[0])


def _max_diff(x, y):
    return float(np.abs(x.astype(np.float64) - y.astype(np.float64)).max())


def test_branch_isolation(fa):
    """Changing branch 2's query and suffix values leaves every other branch's output bit for bit
    unchanged (new random values move branch 2's output by O(0.1))."""
    w = W.make("mid")
    plan = contig_plan(fa, w)
    out, _ = run_contig(plan, to_dev_contig(w), 32)
    rng = np.random.default_rng(3)
    w.q[2] = W.bf16_bits(rng.standard_normal(w.q[2].shape).astype(np.float32))
    w.suffix_v[2, :, :w.suffix_len[2]] = W.bf16_bits(
        rng.standard_normal(w.suffix_v[2, :, :w.suffix_len[2]].shape).astype(np.float32))
    out2, _ = run_contig(plan, to_dev_contig(w), 32)
    scale = max(1.0, float(np.abs(out).max()))
    for b in range(w.n_branches):
        if b != 2:
            assert np.array_equal(out2[b], out[b]), (b, _max_diff(out2[b], out[b]))
        else:
            assert _max_diff(out2[b], out[b]) > 1e-2 * scale


def test_repeatable(fa):
    """Repeated decodes are bit-identical: the slices are dealt to the waves in a fixed order, and
    the first call (which builds its schedule) and the later ones (which take the cached one) run the
    same schedule."""
    w = W.make("mid")
    plan = contig_plan(fa, w)
    dv = to_dev_contig(w)
    a, al = run_contig(plan, dv, 32)
    for _ in range(3):
        b, bl = run_contig(plan, dv, 32)
        assert np.array_equal(a, b), _max_diff(a, b)
        assert np.array_equal(al, bl), _max_diff(al, bl)


def _slot_key_ranges(sl, lens, G):
    """Per row of a slot (fka_plan_slots): the sequence, its prefix key range and its suffix key
    range.  The unit's suffix list holds each sequence's ceil(len / 32) slices in order."""
    out = []
    cs = 0
    for i in range(sl["nseq"]):
        s = sl["seq0"] + i
        L = int(lens[s])
        n = -(-L // 32)
        a, b = max(sl["suffix_begin"], cs), min(sl["suffix_end"], cs + n)
        sr = (32 * (a - cs), min(32 * (b - cs), L)) if b > a else (0, 0)
        for r in range(G):
            out.append((s, (sl["prefix_begin"], sl["prefix_end"]), sr))
        cs += n
    return out


def _check_slot_values(po, pl, slots, info, ref_fn, lens, G, note):
    """Every slot equals the oracle's attention of its rows over their key ranges, and the slots
    of each item tile its prefix and its suffix list exactly."""
    assert len(slots) > 0
    seen = set()
    cover = {}
    for sl in slots:
        assert sl["slot"] not in seen and 0 <= sl["slot"] < info.n_slots
        seen.add(sl["slot"])
        cover.setdefault((sl["seq0"], sl["kv_head"]), []).append(sl)
        g = sl["kv_head"]
        for r, (s, pr, sr) in enumerate(_slot_key_ranges(sl, lens, G)):
            h = g * G + r % G
            what = f"{note} slot {sl['slot']} row {r} seq {s} prefix {pr} suffix {sr}"
            if pr[1] > pr[0] or sr[1] > sr[0]:
                ref, ref_lse = ref_fn(s, h, pr, sr)
                gates.assert_gates(po[sl["slot"], r][None], ref[None], what=what)
                gates.assert_lse(pl[sl["slot"], r][None], np.array([ref_lse]), what=what)
            else:
                assert np.all(po[sl["slot"], r] == 0) and np.isneginf(pl[sl["slot"], r]), what
    for key, sls in cover.items():
        P = sls[0]["prefix_len"]
        pre = sorted((x["prefix_begin"], x["prefix_end"]) for x in sls)
        suf = sorted((x["suffix_begin"], x["suffix_end"]) for x in sls)
        nsuf = sum(-(-int(lens[sls[0]["seq0"] + i]) // 32) for i in range(sls[0]["nseq"]))
        assert pre[0][0] == 0 and pre[-1][1] == P, (key, pre[:3], pre[-3:])
        assert suf[0][0] == 0 and suf[-1][1] == nsuf, (key, suf[:3], suf[-3:])
        for (a0, a1), (b0, b1) in zip(pre, pre[1:]):
            assert a1 == b0, key
        for (a0, a1), (b0, b1) in zip(suf, suf[1:]):
            assert a1 == b0, key


def _check_slots(fa, w, plan, note):
    """Contiguous plan: the first stage's partials against the oracle, slot by slot."""
    info = plan.info()
    dv = to_dev_contig(w)
    N, Hq, d = w.q.shape
    G = Hq // w.spec.n_kv_heads
    po = torch.full((info.n_slots, info.slot_rows, d), float("nan"), device="cuda")
    pl = torch.full((info.n_slots, info.slot_rows), float("nan"), device="cuda")
    plan.partials(dv["q"], dv["prefix_k"], dv["prefix_v"], dv["suffix_k"], dv["suffix_v"], dv["suffix_len"], po, pl)
    torch.cuda.synchronize()
    po, pl = po.cpu().numpy(), pl.cpu().numpy()

    def ref_fn(s, h, pr, sr):
        ref, ref_lse = oracle.decode_contig(w.q, w.prefix_k, w.prefix_v, w.suffix_k, w.suffix_v, w.suffix_len,
                                            w.spec.softmax_scale, prefix_range=pr, suffix_range=sr,
                                            rows=[s * Hq + h])
        return ref[s, h], ref_lse[s, h]

    _check_slot_values(po, pl, plan.slots(w.suffix_len), info, ref_fn, w.suffix_len, G, note)


def _check_slots_paged(fa, w, plan, note):
    """Paged plan: each sequence's prefix and suffix gathered on the host (the oracle's page
    walk) into the contiguous layout, then as for a contiguous plan."""
    info = plan.info()
    dv = to_dev_paged(w)
    S, Hq, d = w.q.shape
    G = Hq // w.spec.n_kv_heads
    po = torch.full((info.n_slots, info.slot_rows, d), float("nan"), device="cuda")
    pl = torch.full((info.n_slots, info.slot_rows), float("nan"), device="cuda")
    plan.partials_paged(dv["q"], dv["k_pool"], dv["v_pool"], dv["page_table"], dv["suffix_len"], po, pl)
    torch.cuda.synchronize()
    po, pl = po.cpu().numpy(), pl.cpu().numpy()
    cache = {}

    def seq_kv(s):
        if s not in cache:
            Lp, L = int(w.seq_prefix_len[s]), int(w.suffix_len[s])
            cache[s] = (Lp, L) + oracle.gather_paged(w.k_pool, w.v_pool, w.page_table, s, Lp, L)
        return cache[s]

    def ref_fn(s, h, pr, sr):
        Lp, L, k, v = seq_kv(s)
        cap = max(L, 1)
        sk = np.full((1, k.shape[0], cap, d), W.BF16_NAN, np.uint16)
        sv = sk.copy()
        sk[0, :, :L], sv[0, :, :L] = k[:, Lp:], v[:, Lp:]
        ref, ref_lse = oracle.decode_contig(w.q[s:s + 1], np.ascontiguousarray(k[:, :Lp]),
                                            np.ascontiguousarray(v[:, :Lp]), sk, sv, np.array([L], np.int32),
                                            w.spec.softmax_scale, prefix_range=pr, suffix_range=sr, rows=[h])
        return ref[0, h], ref_lse[0, h]

    _check_slot_values(po, pl, plan.slots(w.suffix_len), info, ref_fn, w.suffix_len, G, note)


def test_lengths_change_between_calls(fa):
    """Every launch schedules from the lengths it finds on the device: lengths set by the host
    between calls (new ones, empty suffixes, an earlier set again), a partial stage launched in
    between, and repeated calls all match the oracle."""
    w = W.make("mid", steps=0, seed=83)
    plan = contig_plan(fa, w)
    dv = to_dev_contig(w)
    N, Hq, d = w.q.shape
    info = plan.info()
    rng = np.random.default_rng(12)
    # lengths up to the generated ones (positions past them hold NaN on purpose)
    full = w.suffix_len.astype(np.int64)
    sets = [w.suffix_len.copy(), rng.integers(0, full + 1).astype(np.int32), w.suffix_len.copy(),
            np.zeros(N, np.int32), np.minimum(rng.integers(0, 40, N), full).astype(np.int32), w.suffix_len.copy()]
    for i, ln in enumerate(sets):
        print(f"[lengths] set {i}: {ln.tolist()}", flush=True)
        dv["suffix_len"].copy_(torch.from_numpy(ln))
        ref, ref_lse = oracle.decode_contig(w.q, w.prefix_k, w.prefix_v, w.suffix_k, w.suffix_v, ln,
                                            w.spec.softmax_scale)
        for rep in range(3):
            if rep == 1 and i in (1, 4):
                po = torch.empty((info.n_slots, info.slot_rows, d), device="cuda")
                pl = torch.empty((info.n_slots, info.slot_rows), device="cuda")
                plan.partials(dv["q"], dv["prefix_k"], dv["prefix_v"], dv["suffix_k"], dv["suffix_v"],
                              dv["suffix_len"], po, pl)
            out, lse = run_contig(plan, dv, Hq)
            gates.assert_gates(out, ref, what=f"set {i} call {rep}")
            gates.assert_lse(lse, ref_lse, what=f"set {i} call {rep}")
    assert plan.device_error() == 0


@pytest.mark.parametrize("rounds", [0, 5])
def test_partials_stage(fa, rounds):
    """Each first-stage partial equals the oracle's attention over that slot's key ranges."""
    w = W.make("mid", prefix_len=5000, seed=81)
    _check_slots(fa, w, contig_plan(fa, w, rounds=rounds), f"rounds={rounds}")


def test_partials_stage_naive_plan(fa):
    w = W.make("tiny-unscaled", prefix_len=700, suffix_range=(0, 90), seed=82)
    _check_slots(fa, w, contig_plan(fa, w, share_prefix=False), "naive")


@pytest.mark.parametrize("blocks", [3, 16])
def test_partials_stage_few_blocks(fa, blocks):
    """Grids that do not divide the KV heads evenly: blocks straddle two items."""
    w = W.make("mid", prefix_len=3000, seed=84)
    _check_slots(fa, w, contig_plan(fa, w, blocks=blocks), f"blocks={blocks}")


def test_partials_stage_paged(fa):
    """The paged first stage, slot by slot (several groups: the proportional split)."""
    w = _small_paged(seed=91)
    _check_slots_paged(fa, w, paged_plan(fa, w), "paged")


def test_partials_stage_paged_one_group(fa):
    """A paged plan with one group takes the static split."""
    w = W.make(W.CONFIGS["paged"].replace(n_tasks=1, prefix_range=(1500, 1500), suffix_range=(0, 300), seed=92))
    plan = paged_plan(fa, w)
    assert plan.info().static_split == 1
    _check_slots_paged(fa, w, plan, "paged one group")


@pytest.mark.parametrize("d", [64, 128])
def test_lse_merge_stage(fa, d):
    rng = np.random.default_rng(d)
    P, R = 13, 37
    o = rng.standard_normal((P, R, d)).astype(np.float32)
    l = rng.uniform(-30, 30, (P, R)).astype(np.float32)
    l[rng.random((P, R)) < 0.3] = -np.inf
    l[:, 5] = -np.inf           # a row with no keys at all
    o[:, 5] = 0
    out = torch.empty((R, d), device="cuda")
    lse = torch.empty((R,), device="cuda")
    fa.lse_merge(torch.from_numpy(o).cuda(), torch.from_numpy(l).cuda(), out, lse)
    torch.cuda.synchronize()
    ref, ref_lse = oracle.lse_merge(o.transpose(1, 0, 2).astype(np.float64), l.T.astype(np.float64))
    np.testing.assert_allclose(out.cpu().numpy(), ref, rtol=1e-5, atol=1e-5)
    got_lse = lse.cpu().numpy()
    assert np.isneginf(got_lse[5]) and np.array_equal(out.cpu().numpy()[5], np.zeros(d, np.float32))
    fin = np.isfinite(ref_lse)
    np.testing.assert_allclose(got_lse[fin], ref_lse[fin], rtol=1e-6, atol=1e-5)


def _small_paged(headroom=0, seed=90):
    return W.make(W.CONFIGS["paged"].replace(n_tasks=5, prefix_range=(1, 3000), suffix_range=(0, 400),
                                             page_headroom=headroom, seed=seed))


def _random_paged(n, seed):
    rng = np.random.default_rng(seed)
    out = []
    for _ in range(n):
        d = int(rng.choice([64, 128]))
        hkv = int(rng.choice([1, 2, 4, 8]))
        g = int(rng.integers(1, 9))
        nb = int(rng.integers(1, 7))
        while nb * g > 64:
            nb -= 1
        p0 = int(rng.integers(0, 2000))
        s0 = int(rng.integers(0, 300))
        out.append(dict(head_dim=d, n_kv_heads=hkv, n_q_heads=hkv * g, n_branches=nb,
                        n_tasks=int(rng.integers(1, 7)), prefix_range=(p0, p0 + int(rng.integers(0, 3000))),
                        suffix_range=(s0, s0 + int(rng.integers(0, 400))), page_headroom=int(rng.integers(0, 3)),
                        seed=int(rng.integers(1, 1 << 30)), share=bool(rng.integers(0, 4) > 0)))
    return out


@pytest.mark.parametrize("case", _random_paged(8, 4242), ids=lambda c: "d{head_dim}-kv{n_kv_heads}-q{n_q_heads}-b{n_branches}-"
                         "t{n_tasks}-p{prefix_range[0]}_{prefix_range[1]}-{share}".format(**c))
def test_random_paged_shapes(fa, case):
    """Paged parity on seeded random shapes: tasks, branches, GQA group, head_dim, prefix and
    suffix lengths (pages scattered by a random permutation of the pool)."""
    c = dict(case)
    share = c.pop("share")
    w = W.make(W.CONFIGS["paged"].replace(**c))
    print(f"[random paged] {case}", flush=True)
    ref, ref_lse = oracle.decode_workload(w)
    out, lse = run_paged(paged_plan(fa, w, share_prefix=share), to_dev_paged(w))
    gates.assert_gates(out, ref, what="random paged")
    gates.assert_lse(lse, ref_lse, what="random paged")


def test_paged_small_parity_and_naive(fa):
    w = _small_paged()
    ref, ref_lse = oracle.decode_workload(w)
    dv = to_dev_paged(w)
    for share in (True, False):
        out, lse = run_paged(paged_plan(fa, w, share_prefix=share), dv)
        gates.assert_gates(out, ref, what=f"paged share={share}")
        gates.assert_lse(lse, ref_lse, what=f"paged share={share}")


def test_paged_equals_contiguous_on_same_data(fa):
    """The paged path and the contiguous path agree on one task's gathered data."""
    w = _small_paged(seed=91)
    dv = to_dev_paged(w)
    outp, _ = run_paged(paged_plan(fa, w), dv)
    t = 2
    s0, s1 = int(w.group_start[t]), int(w.group_start[t + 1])
    Lp = int(w.prefix_len[t])
    Ls = w.suffix_len[s0:s1]
    cap = max(1, int(Ls.max()))
    K = np.full((s1 - s0, w.spec.n_kv_heads, cap, w.spec.head_dim), W.BF16_NAN, np.uint16)
    V = K.copy()
    pk = pv = None
    for j, i in enumerate(range(s0, s1)):
        ko, vo = oracle.gather_paged(w.k_pool, w.v_pool, w.page_table, i, Lp, int(Ls[j]))
        pk, pv = ko[:, :Lp], vo[:, :Lp]
        K[j, :, :Ls[j]] = ko[:, Lp:]
        V[j, :, :Ls[j]] = vo[:, Lp:]
    cw = W.ContigWorkload(w.spec.replace(paged=False, n_branches=s1 - s0), w.q[s0:s1], np.ascontiguousarray(pk),
                          np.ascontiguousarray(pv), K, V, Ls.astype(np.int32))
    outc, _ = run_contig(contig_plan(fa, cw), to_dev_contig(cw), w.spec.n_q_heads)
    gates.assert_gates(outp[s0:s1], outc.astype(np.float64), what="paged vs contiguous")


def test_gather_bit_exact(fa):
    w = _small_paged(seed=92)
    plan = paged_plan(fa, w)
    dv = to_dev_paged(w)
    for i in range(w.n_seqs):
        t = i // w.spec.n_branches
        Lp, Ls = int(w.prefix_len[t]), int(w.suffix_len[i])
        L = Lp + Ls
        ko = torch.empty((w.spec.n_kv_heads, max(L, 1), w.spec.head_dim), dtype=torch.bfloat16, device="cuda")
        vo = torch.empty_like(ko)
        plan.gather_paged(i, dv["k_pool"], dv["v_pool"], dv["page_table"], L, ko, vo)
        torch.cuda.synchronize()
        rk, rv = oracle.gather_paged(w.k_pool, w.v_pool, w.page_table, i, Lp, Ls)
        assert np.array_equal(ko.view(torch.int16).cpu().numpy().view(np.uint16)[:, :L], rk)
        assert np.array_equal(vo.view(torch.int16).cpu().numpy().view(np.uint16)[:, :L], rv)


def test_gather_bit_exact_full_paged_sample(fa):
    w = W.make("paged")
    plan = paged_plan(fa, w)
    dv = to_dev_paged(w)
    for i in (0, 7, 41, 79):
        t = i // w.spec.n_branches
        Lp, Ls = int(w.prefix_len[t]), int(w.suffix_len[i])
        L = Lp + Ls
        ko = torch.empty((w.spec.n_kv_heads, L, w.spec.head_dim), dtype=torch.bfloat16, device="cuda")
        vo = torch.empty_like(ko)
        plan.gather_paged(i, dv["k_pool"], dv["v_pool"], dv["page_table"], L, ko, vo)
        torch.cuda.synchronize()
        rk, rv = oracle.gather_paged(w.k_pool, w.v_pool, w.page_table, i, Lp, Ls)
        assert np.array_equal(ko.view(torch.int16).cpu().numpy().view(np.uint16), rk)
        assert np.array_equal(vo.view(torch.int16).cpu().numpy().view(np.uint16), rv)


def test_paged_append_then_decode(fa):
    w = _small_paged(headroom=40, seed=93)
    plan = paged_plan(fa, w)
    dv = to_dev_paged(w)
    rng = np.random.default_rng(4)
    S, Hkv, d = w.n_seqs, w.spec.n_kv_heads, w.spec.head_dim
    P = w.spec.page_size
    for step in range(20):
        kn = W.bf16_bits(rng.standard_normal((S, Hkv, d)).astype(np.float32))
        vn = W.bf16_bits(rng.standard_normal((S, Hkv, d)).astype(np.float32))
        plan.append_paged(dev_bf16(kn), dev_bf16(vn), dv["k_pool"], dv["v_pool"], dv["page_table"], dv["suffix_len"])
        for i in range(S):
            t = i // w.spec.n_branches
            u = int(w.suffix_len[i])
            page = w.page_table[i, -(-int(w.prefix_len[t]) // P) + u // P]
            w.k_pool[page, :, u % P] = kn[i]
            w.v_pool[page, :, u % P] = vn[i]
            w.suffix_len[i] = u + 1
    torch.cuda.synchronize()
    assert np.array_equal(dv["suffix_len"].cpu().numpy(), w.suffix_len)
    assert np.array_equal(dv["k_pool"].view(torch.int16).cpu().numpy().view(np.uint16), w.k_pool)
    ref, _ = oracle.decode_workload(w)
    out, _ = run_paged(plan, dv)
    gates.assert_gates(out, ref, what="paged after appends")
    assert plan.device_error() == 0


def test_append_past_capacity_is_flagged_not_written(fa):
    w = W.make("tiny", suffix_range=(0, 8))
    plan = contig_plan(fa, w, max_suffix_len=8)
    dv = to_dev_contig(w)
    dv["suffix_len"].fill_(8)
    before = dv["suffix_k"].clone()
    kn = torch.zeros((w.n_branches, 2, 64), dtype=torch.bfloat16, device="cuda")
    plan.append(kn, kn, dv["suffix_k"], dv["suffix_v"], dv["suffix_len"])
    torch.cuda.synchronize()
    assert torch.equal(dv["suffix_len"].cpu(), torch.full((w.n_branches,), 8, dtype=torch.int32))
    assert torch.equal(before.view(torch.int16), dv["suffix_k"].view(torch.int16))
    assert plan.device_error() & 2
    assert plan.device_error() == 0   # reading clears the flag


def test_suffix_length_above_bound_is_clamped_and_flagged(fa):
    w = W.make("tiny", suffix_range=(10, 20))
    plan = contig_plan(fa, w, max_suffix_len=12)
    dv = to_dev_contig(w)
    dv["suffix_len"].fill_(40)
    out, _ = run_contig(plan, dv, 8)
    w.suffix_len[:] = 12
    ref, _ = oracle.decode_workload(w)
    gates.assert_gates(out, ref, what="clamped lengths")
    assert plan.device_error() & 1


def _close_to_unfused(oa, la, ob, lb, what):
    """The fused step and append + decode compute the same sums with different splits of the keys
    (appending one token moves the balanced schedule), so they agree up to rounding: P carries
    ~2^-17 relative error per element (hi + lo bf16 terms), which bounds the output difference
    well below 1e-4 of the output scale; lse agrees to fp32 rounding of the sums."""
    scale = max(1.0, float(ob.abs().max()))
    d = float((oa - ob).abs().max())
    dl = float((la - lb).abs().max())
    print(f"[fused] {what}: max|fused - unfused| = {d:.3g} (scale {scale:.3g}), lse {dl:.3g}", flush=True)
    assert d <= 1e-4 * scale, f"{what}: {d}"
    assert dl <= 1e-5, f"{what}: lse {dl}"


def test_fused_step_equals_append_then_decode(fa):
    """fka_fork_step (append fused into the decode) matches append + decode: identical caches and
    lengths; the output matches the oracle on the appended state and the unfused output up to
    rounding (the new token is merged as its own part)."""
    w = W.make("mid", steps=8)
    plan = contig_plan(fa, w)
    a, b = to_dev_contig(w), to_dev_contig(w)
    N, Hq, d = w.q.shape
    oa, la = torch.empty((N, Hq, d), device="cuda"), torch.empty((N, Hq), device="cuda")
    ob, lb = torch.empty_like(oa), torch.empty_like(la)
    kn, vn, qn = dev_bf16(w.step_k), dev_bf16(w.step_v), dev_bf16(w.step_q)
    for t in range(8):
        plan.step(qn[t], kn[t], vn[t], a["prefix_k"], a["prefix_v"], a["suffix_k"], a["suffix_v"], a["suffix_len"],
                  oa, la)
        plan.append(kn[t], vn[t], b["suffix_k"], b["suffix_v"], b["suffix_len"])
        plan.decode(qn[t], b["prefix_k"], b["prefix_v"], b["suffix_k"], b["suffix_v"], b["suffix_len"], ob, lb)
        torch.cuda.synchronize()
        _close_to_unfused(oa, la, ob, lb, f"contiguous step {t}")
        if t in (0, 7):
            sk = b["suffix_k"].view(torch.int16).cpu().numpy().view(np.uint16)
            sv = b["suffix_v"].view(torch.int16).cpu().numpy().view(np.uint16)
            ln = b["suffix_len"].cpu().numpy()
            ref, ref_lse = oracle.decode_contig(w.step_q[t], w.prefix_k, w.prefix_v, sk, sv, ln, w.spec.softmax_scale)
            gates.assert_gates(oa.cpu().numpy(), ref, what=f"fused step {t}")
            gates.assert_lse(la.cpu().numpy(), ref_lse, what=f"fused step {t}")
    assert torch.equal(a["suffix_len"], b["suffix_len"])
    assert torch.equal(a["suffix_k"].view(torch.int16), b["suffix_k"].view(torch.int16))
    assert torch.equal(a["suffix_v"].view(torch.int16), b["suffix_v"].view(torch.int16))
    assert plan.device_error() == 0


def test_fused_step_paged_equals_append_then_decode(fa):
    w = _small_paged(headroom=24, seed=94)
    plan = paged_plan(fa, w)
    a, b = to_dev_paged(w), to_dev_paged(w)
    S, Hq, d = w.q.shape
    rng = np.random.default_rng(5)
    oa, la = torch.empty((S, Hq, d), device="cuda"), torch.empty((S, Hq), device="cuda")
    ob, lb = torch.empty_like(oa), torch.empty_like(la)
    for t in range(20):
        kn_h = W.bf16_bits(rng.standard_normal((S, w.spec.n_kv_heads, d)).astype(np.float32))
        vn_h = W.bf16_bits(rng.standard_normal((S, w.spec.n_kv_heads, d)).astype(np.float32))
        q_h = W.bf16_bits(rng.standard_normal((S, Hq, d)).astype(np.float32))
        kn, vn, q = dev_bf16(kn_h), dev_bf16(vn_h), dev_bf16(q_h)
        plan.step_paged(q, kn, vn, a["k_pool"], a["v_pool"], a["page_table"], a["suffix_len"], oa, la)
        plan.append_paged(kn, vn, b["k_pool"], b["v_pool"], b["page_table"], b["suffix_len"])
        plan.decode_paged(q, b["k_pool"], b["v_pool"], b["page_table"], b["suffix_len"], ob, lb)
        torch.cuda.synchronize()
        _close_to_unfused(oa, la, ob, lb, f"paged step {t}")
        if t in (0, 19):
            kp = b["k_pool"].view(torch.int16).cpu().numpy().view(np.uint16)
            vp = b["v_pool"].view(torch.int16).cpu().numpy().view(np.uint16)
            ln = b["suffix_len"].cpu().numpy()
            ref, ref_lse = oracle.decode_paged(q_h, kp, vp, w.page_table, w.seq_prefix_len, ln, w.spec.softmax_scale)
            gates.assert_gates(oa.cpu().numpy(), ref, what=f"fused paged step {t}")
            gates.assert_lse(la.cpu().numpy(), ref_lse, what=f"fused paged step {t}")
    assert torch.equal(a["suffix_len"], b["suffix_len"])
    assert torch.equal(a["k_pool"].view(torch.int16), b["k_pool"].view(torch.int16))
    assert plan.device_error() == 0


def test_fused_step_at_capacity_is_flagged(fa):
    w = W.make("tiny", suffix_range=(8, 8))          # every suffix already at the bound
    plan = contig_plan(fa, w, max_suffix_len=8)
    dv = to_dev_contig(w)
    kn = torch.zeros((w.n_branches, 2, 64), dtype=torch.bfloat16, device="cuda")
    out = torch.empty((w.n_branches, 8, 64), device="cuda")
    plan.step(dv["q"], kn, kn, dv["prefix_k"], dv["prefix_v"], dv["suffix_k"], dv["suffix_v"], dv["suffix_len"], out)
    torch.cuda.synchronize()
    assert torch.equal(dv["suffix_len"].cpu(), torch.full((w.n_branches,), 8, dtype=torch.int32))
    assert plan.device_error() & 2
    ref, _ = oracle.decode_workload(w)       # the full buffers, without the token that did not fit
    gates.assert_gates(out.cpu().numpy(), ref, what="step at capacity")


def test_nan_input_propagates_to_its_branch_only(fa):
    w = W.make("mid", seed=95)
    w.suffix_v[3, 2, 5] = W.BF16_NAN            # one value row of branch 3, KV head 2
    out, lse = run_contig(contig_plan(fa, w), to_dev_contig(w), 32)
    G = w.spec.group
    bad = np.zeros(out.shape[:2], bool)
    bad[3, 2 * G:3 * G] = True
    assert np.all(np.isnan(out[bad]).any(axis=-1))
    assert np.all(np.isfinite(out[~bad]))
    ref, _ = oracle.decode_workload(w)
    gates.assert_gates(out[~bad], ref[~bad], what="rows without the NaN")


def test_graph_replay_matches_eager(fa):
    """The benchmark launches its timed steps as a captured HIP graph.  Fused steps captured once
    and replayed several times (with the lengths reset, and eager work and synchronisations in
    between) give, in every replay, exactly what the same steps give when launched one by one."""
    w = W.make("mid", steps=6, seed=96)
    plan = contig_plan(fa, w)
    dv = to_dev_contig(w)
    N, Hq, d = w.q.shape
    kn, vn, qn = dev_bf16(w.step_k), dev_bf16(w.step_v), dev_bf16(w.step_q)
    len0 = dv["suffix_len"].clone()
    outs = [torch.empty((N, Hq, d), device="cuda") for _ in range(6)]
    lses = [torch.empty((N, Hq), device="cuda") for _ in range(6)]

    def steps():
        for t in range(6):
            plan.step(qn[t], kn[t], vn[t], dv["prefix_k"], dv["prefix_v"], dv["suffix_k"], dv["suffix_v"],
                      dv["suffix_len"], outs[t], lses[t])

    steps()
    torch.cuda.synchronize()
    ref = [o.cpu().numpy().copy() for o in outs]
    ref_lse = [x.cpu().numpy().copy() for x in lses]
    ref_k = dv["suffix_k"].view(torch.int16).cpu().numpy().copy()
    dv["suffix_len"].copy_(len0)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        steps()
    torch.cuda.synchronize()
    for rep in range(3):
        dv["suffix_len"].copy_(len0)
        for o in outs:
            o.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        for t in range(6):
            assert np.array_equal(outs[t].cpu().numpy(), ref[t]), f"replay {rep} step {t}"
            assert np.array_equal(lses[t].cpu().numpy(), ref_lse[t]), f"replay {rep} step {t} lse"
        assert np.array_equal(dv["suffix_k"].view(torch.int16).cpu().numpy(), ref_k)
        assert np.array_equal(dv["suffix_len"].cpu().numpy(), (len0 + 6).cpu().numpy())
        _ = torch.randn(1000, device="cuda").sum().item()  # eager work between replays
    assert plan.device_error() == 0
