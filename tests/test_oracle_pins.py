"""Pins of the fp64 oracle to facts that do not come from the oracle itself.

The paper prints no attention values, so the oracle is pinned by
  * brute force: 50-digit mpmath evaluation of sum_j e^{s_j} v_j / sum_j e^{s_j}
    (no max subtraction, a different formulation) on tiny inputs;
  * a library special case: torch's CPU fp64 scaled_dot_product_attention per
    branch over the materialised [prefix ; own suffix], K/V heads expanded with
    repeat_interleave (which fixes the grouped-query mapping h -> h // G);
  * closed forms (constant keys, zero query, one and two keys, empty context);
  * invariants of the method: identical queries with empty suffixes give
    identical branch outputs, branches do not see each other (Sec. 3.2, 3.3),
    chunked attention merged by log-sum-exp equals the unchunked result, and
    the paged walk equals the contiguous result on the same logical data;
  * mutation checks: plausible mistakes (dropped suffix, dropped tile, swapped
    branches, wrong head mapping, missing scale) fail the tolerance gates.
"""
import math
import zlib

import numpy as np
import pytest
import torch

import oracle
from paper_2608_13667_amd import workloads as W
from tests import gates


def _problem(rng, N=3, Hq=4, Hkv=2, d=8, Lp=7, lens=(0, 3, 5), cap=None, scale=1.0):
    lens = np.asarray(lens, np.int32)
    cap = int(cap or max(1, lens.max(initial=0)))
    f = lambda *s: W.bf16_bits((rng.standard_normal(s) * scale).astype(np.float32))
    sk = np.full((N, Hkv, cap, d), W.BF16_NAN, np.uint16)
    sv = np.full((N, Hkv, cap, d), W.BF16_NAN, np.uint16)
    for b in range(N):
        sk[b, :, :lens[b]] = f(Hkv, int(lens[b]), d)
        sv[b, :, :lens[b]] = f(Hkv, int(lens[b]), d)
    return dict(q=f(N, Hq, d), prefix_k=f(Hkv, Lp, d), prefix_v=f(Hkv, Lp, d), suffix_k=sk, suffix_v=sv,
                suffix_len=lens)


def _run(p, scale, **kw):
    return oracle.decode_contig(p["q"], p["prefix_k"], p["prefix_v"], p["suffix_k"], p["suffix_v"],
                                p["suffix_len"], scale, **kw)


def _f(bits):
    return W.bf16_to_f32(bits).astype(np.float64)


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    x = (rng.standard_normal(1 << 16) * np.exp(rng.uniform(-20, 20, 1 << 16))).astype(np.float32)
    # include exact ties and values on both sides of them
    x[:4] = np.array([1.00390625, 1.01171875, -1.00390625, 3.0], np.float32)
    ref = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(W.bf16_bits(x), ref)


@pytest.mark.parametrize("case", [
    dict(N=1, Hq=1, Hkv=1, d=4, Lp=1, lens=(0,)),
    dict(N=3, Hq=4, Hkv=2, d=8, Lp=7, lens=(0, 3, 5)),
    dict(N=5, Hq=8, Hkv=2, d=16, Lp=33, lens=(2, 0, 9, 1, 4)),
    dict(N=2, Hq=3, Hkv=3, d=16, Lp=0, lens=(4, 6)),
    dict(N=4, Hq=4, Hkv=1, d=8, Lp=64, lens=(0, 0, 1, 0)),
])
def test_brute_force_mpmath(case):
    mp = pytest.importorskip("mpmath")
    mp.mp.dps = 50
    rng = np.random.default_rng(zlib.crc32(repr(sorted(case.items())).encode()))  # the same inputs in every run
    p = _problem(rng, **case)
    d = case["d"]
    scale = 1.0 / math.sqrt(d)
    out, lse = _run(p, scale)
    N, Hq, Hkv = case["N"], case["Hq"], case["Hkv"]
    G = Hq // Hkv
    qf, pk, pv, sk, sv = (_f(p[k]) for k in ("q", "prefix_k", "prefix_v", "suffix_k", "suffix_v"))
    for b in range(N):
        for h in range(Hq):
            keys = [pk[h // G, j] for j in range(case["Lp"])] + [sk[b, h // G, u] for u in range(p["suffix_len"][b])]
            vals = [pv[h // G, j] for j in range(case["Lp"])] + [sv[b, h // G, u] for u in range(p["suffix_len"][b])]
            den = mp.mpf(0)
            num = [mp.mpf(0)] * d
            sc = mp.mpf(1) / mp.sqrt(d)
            for kk, vv in zip(keys, vals):
                e = mp.exp(sc * mp.fsum(mp.mpf(float(a)) * mp.mpf(float(c)) for a, c in zip(qf[b, h], kk)))
                den += e
                num = [n_ + e * mp.mpf(float(v)) for n_, v in zip(num, vv)]
            for c in range(d):
                assert abs(out[b, h, c] - float(num[c] / den)) <= 1e-13 * max(1.0, abs(float(num[c] / den)))
            assert abs(lse[b, h] - float(mp.log(den))) <= 1e-13 * max(1.0, abs(float(mp.log(den))))


@pytest.mark.parametrize("name,Lp", [("tiny", None), ("tiny-unscaled", None), ("mid", 1024)])
def test_torch_sdpa_fp64(name, Lp):
    spec = W.CONFIGS[name]
    if Lp is not None:
        spec = spec.replace(prefix_len=Lp)
    w = W.make(spec)
    out, _ = oracle.decode_workload(w)
    G = spec.group
    q = torch.from_numpy(W.bf16_to_f32(w.q).astype(np.float64))
    for b in range(w.n_branches):
        L = int(w.suffix_len[b])
        K = np.concatenate([w.prefix_k, w.suffix_k[b, :, :L]], axis=1)
        V = np.concatenate([w.prefix_v, w.suffix_v[b, :, :L]], axis=1)
        Kt = torch.from_numpy(W.bf16_to_f32(K).astype(np.float64)).repeat_interleave(G, dim=0)
        Vt = torch.from_numpy(W.bf16_to_f32(V).astype(np.float64)).repeat_interleave(G, dim=0)
        ref = torch.nn.functional.scaled_dot_product_attention(
            q[b][:, None, :], Kt, Vt, scale=spec.softmax_scale)[:, 0, :].numpy()
        np.testing.assert_allclose(out[b], ref, rtol=1e-12, atol=1e-14)


def test_constant_keys_give_mean_of_values():
    rng = np.random.default_rng(1)
    p = _problem(rng, N=3, Hq=4, Hkv=2, d=8, Lp=20, lens=(0, 5, 11))
    k0 = p["prefix_k"][:, :1, :]
    p["prefix_k"][:] = k0
    for b in range(3):
        p["suffix_k"][b, :, :p["suffix_len"][b]] = k0
    scale = 0.37
    out, lse = _run(p, scale)
    pv, sv, qf = _f(p["prefix_v"]), _f(p["suffix_v"]), _f(p["q"])
    for b in range(3):
        L = p["suffix_len"][b]
        for h in range(4):
            g = h // 2
            ctx = np.concatenate([pv[g], sv[b, g, :L]])
            np.testing.assert_allclose(out[b, h], ctx.mean(axis=0), rtol=1e-13, atol=1e-15)
            s0 = scale * float(np.dot(qf[b, h], _f(k0[g, 0])))
            assert abs(lse[b, h] - (s0 + math.log(20 + L))) <= 1e-12


def test_zero_query_gives_mean_of_values():
    rng = np.random.default_rng(2)
    p = _problem(rng, N=2, Hq=2, Hkv=1, d=8, Lp=9, lens=(3, 0))
    p["q"][:] = 0
    out, lse = _run(p, 0.5)
    pv, sv = _f(p["prefix_v"]), _f(p["suffix_v"])
    np.testing.assert_allclose(out[0, 0], np.concatenate([pv[0], sv[0, 0, :3]]).mean(0), rtol=1e-13)
    np.testing.assert_allclose(out[1, 1], pv[0].mean(0), rtol=1e-13)
    assert abs(lse[0, 0] - math.log(12)) < 1e-14 and abs(lse[1, 0] - math.log(9)) < 1e-14


def test_one_and_two_keys():
    rng = np.random.default_rng(3)
    p = _problem(rng, N=2, Hq=1, Hkv=1, d=16, Lp=1, lens=(0, 1))
    scale = 0.25
    out, lse = _run(p, scale)
    qf, pk, pv, sk, sv = (_f(p[k]) for k in ("q", "prefix_k", "prefix_v", "suffix_k", "suffix_v"))
    # one key: the value itself, exactly
    assert np.array_equal(out[0, 0], pv[0, 0])
    assert abs(lse[0, 0] - scale * float(np.dot(qf[0, 0], pk[0, 0]))) < 1e-14
    # two keys: logistic weights
    s0 = scale * float(np.dot(qf[1, 0], pk[0, 0]))
    s1 = scale * float(np.dot(qf[1, 0], sk[1, 0, 0]))
    w0 = 1.0 / (1.0 + math.exp(s1 - s0))
    np.testing.assert_allclose(out[1, 0], w0 * pv[0, 0] + (1 - w0) * sv[1, 0, 0], rtol=1e-13, atol=1e-15)


def test_empty_context():
    rng = np.random.default_rng(4)
    p = _problem(rng, N=2, Hq=2, Hkv=1, d=8, Lp=0, lens=(0, 2))
    out, lse = _run(p, 0.3)
    assert np.array_equal(out[0], np.zeros((2, 8))) and np.all(np.isneginf(lse[0]))
    assert np.all(np.isfinite(out[1])) and np.all(np.isfinite(lse[1]))


def test_identical_queries_empty_suffixes_identical_outputs():
    w = W.make("mid", prefix_len=512, suffix_range=(0, 0))
    w.q[:] = w.q[0:1]
    out, lse = oracle.decode_workload(w)
    for b in range(1, w.n_branches):
        assert np.array_equal(out[b], out[0]) and np.array_equal(lse[b], lse[0])


def test_branches_do_not_see_each_other():
    w = W.make("tiny-unscaled")
    out, lse = oracle.decode_workload(w)
    rng = np.random.default_rng(5)
    # perturb branch 2's query and suffix, and lengthen it
    w.q[2] = W.bf16_bits(rng.standard_normal(w.q[2].shape).astype(np.float32))
    w.suffix_k[2] = W.bf16_bits(rng.standard_normal(w.suffix_k[2].shape).astype(np.float32))
    w.suffix_len[2] = w.suffix_cap
    out2, lse2 = oracle.decode_workload(w)
    for b in range(w.n_branches):
        if b != 2:
            assert np.array_equal(out2[b], out[b]) and np.array_equal(lse2[b], lse[b])
    assert not np.allclose(out2[2], out[2])


@pytest.mark.parametrize("seed", [0, 1, 2])
def test_chunked_merge_equals_unchunked(seed):
    rng = np.random.default_rng(100 + seed)
    Lp, cap = 300, 40
    p = _problem(rng, N=3, Hq=4, Hkv=2, d=16, Lp=Lp, lens=(0, 17, 40), cap=cap)
    scale = 0.25
    full, full_lse = _run(p, scale)
    # random chunk boundaries over the prefix and the suffix, including empty chunks
    pb = np.sort(np.concatenate([[0, Lp], rng.integers(0, Lp + 1, 5), [17, 17]]))
    sb = np.sort(np.concatenate([[0, cap], rng.integers(0, cap + 1, 3)]))
    parts_o, parts_l = [], []
    for lo, hi in zip(pb[:-1], pb[1:]):
        o, l = _run(p, scale, prefix_range=(lo, hi), suffix_range=(0, 0))
        parts_o.append(o), parts_l.append(l)
    for lo, hi in zip(sb[:-1], sb[1:]):
        o, l = _run(p, scale, prefix_range=(0, 0), suffix_range=(lo, hi))
        parts_o.append(o), parts_l.append(l)
    po = np.stack(parts_o, axis=2).reshape(12, len(parts_o), 16)
    pl = np.stack(parts_l, axis=2).reshape(12, len(parts_l))
    m, ml = oracle.lse_merge(po, pl)
    np.testing.assert_allclose(m.reshape(full.shape), full, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(ml.reshape(full_lse.shape), full_lse, rtol=1e-12, atol=1e-14)


def test_merge_of_empty_parts():
    o = np.zeros((2, 3, 4))
    l = np.full((2, 3), -np.inf)
    o[1, 1] = [1, 2, 3, 4]
    l[1, 1] = 0.5
    m, ml = oracle.lse_merge(o, l)
    assert np.array_equal(m[0], np.zeros(4)) and np.isneginf(ml[0])
    assert np.array_equal(m[1], o[1, 1]) and ml[1] == 0.5


def test_prefix_order_does_not_matter():
    rng = np.random.default_rng(6)
    p = _problem(rng, N=2, Hq=4, Hkv=2, d=16, Lp=200, lens=(3, 30))
    out, lse = _run(p, 0.25)
    perm = rng.permutation(200)
    p["prefix_k"] = p["prefix_k"][:, perm]
    p["prefix_v"] = p["prefix_v"][:, perm]
    out2, lse2 = _run(p, 0.25)
    np.testing.assert_allclose(out2, out, rtol=1e-13, atol=1e-15)
    np.testing.assert_allclose(lse2, lse, rtol=1e-13)


def _grid_values(rng, shape):
    """bf16-exact values k/8, |k| <= 16, so that adding 1 stays exact."""
    return W.bf16_bits((rng.integers(-16, 17, shape) / 8.0).astype(np.float32))


def test_value_offset_shifts_output_and_key_offset_does_nothing():
    rng = np.random.default_rng(7)
    p = _problem(rng, N=2, Hq=2, Hkv=1, d=8, Lp=50, lens=(6, 0), cap=6)
    for k in ("prefix_k", "prefix_v"):
        p[k] = _grid_values(rng, p[k].shape)
    p["suffix_k"][0, :, :6] = _grid_values(rng, (1, 6, 8))
    p["suffix_v"][0, :, :6] = _grid_values(rng, (1, 6, 8))
    out, lse = _run(p, 0.3)
    plus1 = lambda bits: W.bf16_bits((W.bf16_to_f32(bits) + 1.0).astype(np.float32))
    pv = dict(p, prefix_v=plus1(p["prefix_v"]), suffix_v=plus1(p["suffix_v"]))
    out_v, _ = _run(pv, 0.3)
    np.testing.assert_allclose(out_v, out + 1.0, rtol=0, atol=1e-14)
    pk = dict(p, prefix_k=plus1(p["prefix_k"]), suffix_k=plus1(p["suffix_k"]))
    out_k, lse_k = _run(pk, 0.3)
    np.testing.assert_allclose(out_k, out, rtol=1e-13, atol=1e-15)
    # every score moved by scale * sum(q): the log-sum-exp moves by the same amount
    shift = 0.3 * _f(p["q"]).sum(-1)
    np.testing.assert_allclose(lse_k, lse + shift, rtol=1e-13, atol=1e-13)


def test_grouped_heads_equal_duplicated_kv_heads():
    rng = np.random.default_rng(8)
    p = _problem(rng, N=2, Hq=6, Hkv=2, d=8, Lp=30, lens=(4, 7), cap=7)
    out, lse = _run(p, 0.4)
    rep = lambda a, ax: np.repeat(a, 3, axis=ax)
    q1 = dict(p, prefix_k=rep(p["prefix_k"], 0), prefix_v=rep(p["prefix_v"], 0),
              suffix_k=rep(p["suffix_k"], 1), suffix_v=rep(p["suffix_v"], 1))
    out1, lse1 = _run(q1, 0.4)
    assert np.array_equal(out1, out) and np.array_equal(lse1, lse)


def test_paged_walk_equals_contiguous():
    spec = W.CONFIGS["paged"].replace(n_tasks=3, prefix_range=(1, 70), suffix_range=(0, 40), n_kv_heads=2,
                                      n_q_heads=8, head_dim=64)
    w = W.make(spec)
    out, lse = oracle.decode_workload(w)
    P = spec.page_size
    for i in range(w.n_seqs):
        t = i // spec.n_branches
        Lp, Ls = int(w.prefix_len[t]), int(w.suffix_len[i])
        # independent gather with numpy fancy indexing
        pos = np.arange(Lp + Ls)
        pidx = np.where(pos < Lp, pos // P, -(-Lp // P) + (pos - Lp) // P)
        slot = np.where(pos < Lp, pos % P, (pos - Lp) % P)
        pages = w.page_table[i, pidx]
        K = w.k_pool[pages, :, slot].transpose(1, 0, 2)
        V = w.v_pool[pages, :, slot].transpose(1, 0, 2)
        ko, vo = oracle.gather_paged(w.k_pool, w.v_pool, w.page_table, i, Lp, Ls)
        assert np.array_equal(ko, K) and np.array_equal(vo, V)
        c_out, c_lse = oracle.decode_contig(w.q[i:i + 1], K[:, :Lp], V[:, :Lp], K[None, :, Lp:], V[None, :, Lp:],
                                            np.array([Ls], np.int32), spec.softmax_scale)
        assert np.array_equal(c_out[0], out[i]) and np.array_equal(c_lse[0], lse[i])


# ---- mutation checks: the gates must reject plausible mistakes -------------------------------

@pytest.fixture(scope="module", params=["tiny-unscaled", "mid"])
def ref_case(request):
    w = W.make(request.param)
    out, lse = oracle.decode_workload(w)
    return w, out, lse


def test_gates_accept_the_oracle_itself(ref_case):
    w, out, _ = ref_case
    assert gates.passes(out.astype(np.float32), out)


def test_mutation_dropped_suffix_fails(ref_case):
    w, out, _ = ref_case
    bad, _ = oracle.decode_contig(w.q, w.prefix_k, w.prefix_v, w.suffix_k, w.suffix_v, np.zeros_like(w.suffix_len),
                                  w.spec.softmax_scale)
    assert not gates.passes(bad, out)


def test_mutation_dropped_prefix_tile_fails(ref_case):
    w, out, _ = ref_case
    bad, _ = oracle.decode_contig(w.q, w.prefix_k, w.prefix_v, w.suffix_k, w.suffix_v, w.suffix_len,
                                  w.spec.softmax_scale, prefix_range=(64, w.prefix_len))
    assert not gates.passes(bad, out)


def test_mutation_swapped_branches_fails(ref_case):
    w, out, _ = ref_case
    bad = out[[1, 0] + list(range(2, w.n_branches))]
    assert not gates.passes(bad, out)


def test_mutation_wrong_head_mapping_fails(ref_case):
    w, out, _ = ref_case
    Hq, Hkv = w.spec.n_q_heads, w.spec.n_kv_heads
    bad = np.empty_like(out)
    for h in range(Hq):
        g = h % Hkv   # the mistake: interleaved instead of contiguous groups
        o, _ = oracle.decode_contig(w.q[:, h:h + 1], w.prefix_k[g:g + 1], w.prefix_v[g:g + 1],
                                    w.suffix_k[:, g:g + 1], w.suffix_v[:, g:g + 1], w.suffix_len, w.spec.softmax_scale)
        bad[:, h] = o[:, 0]
    assert not gates.passes(bad, out)


def test_mutation_missing_scale_fails(ref_case):
    w, out, _ = ref_case
    bad, _ = oracle.decode_contig(w.q, w.prefix_k, w.prefix_v, w.suffix_k, w.suffix_v, w.suffix_len, 1.0)
    assert not gates.passes(bad, out)


@pytest.mark.parametrize("name", ["tiny", "mid", "long", "very-long", "onset"])
def test_workload_lengths(name):
    """Suffix lengths are integers drawn inclusively from the stated ranges; the fork-onset
    workload's main sequence draws from its own (long) range after the branches, so the branch
    draws match those of the same spec without it."""
    spec = W.CONFIGS[name]
    w = W.make(spec.replace(steps=0))
    lo, hi = spec.suffix_range
    first = 0 if spec.main_suffix_range is None else 1
    assert all(lo <= int(L) <= hi for L in w.suffix_len[first:])
    if spec.main_suffix_range is not None:
        mlo, mhi = spec.main_suffix_range
        assert mlo <= int(w.suffix_len[0]) <= mhi
        base = W.make(spec.replace(main_suffix_range=None, steps=0, prefix_len=16))
        assert np.array_equal(base.suffix_len[1:], w.suffix_len[1:])
    assert w.suffix_k.shape[2] >= int(w.suffix_len.max())


def test_oracle_refuses_lengths_outside_the_buffer():
    """A suffix holds 0..cap tokens; the oracle defines nothing else (no clamping by itself)."""
    rng = np.random.default_rng(3)
    p = _problem(rng, N=2, Hq=2, Hkv=1, d=4, Lp=3, lens=(1, 2))
    for bad in ((1, p["suffix_k"].shape[2] + 1), (-1, 0)):
        with pytest.raises(ValueError, match="suffix length"):
            oracle.decode_contig(p["q"], p["prefix_k"], p["prefix_v"], p["suffix_k"], p["suffix_v"],
                                 np.array(bad, np.int32), 0.5)
