"""Seeded synthetic inputs for fork-aware decode attention.

This module draws random numbers and lays them out; it performs none of the
attention arithmetic.  The oracle tests and the HIP path consume the same
arrays, so it is the one module both sides import.

Workload shape (paper, Sec. 3.2 Overview and Sec. 3.3 Forking via Trajectory
Continuation): at the fork instant every branch holds the same snapshot of the
history H_t followed by the thought R_t, plus its own short continuation.  The
main thread and the four auxiliary branches decode concurrently, so one decode
step has N = 5 sequences, each contributing one new query token, all reading one
shared prefix K/V and each reading its own suffix K/V.  The paper's benchmark
trajectories (SWE-Bench Pro, Terminal-Bench 2.1, tau^3-bench) are not used;
these synthetic shapes stand in for them.

Recipe (all draws from ``numpy.random.Generator(PCG64)``):

* ``SeedSequence(seed).spawn(9)`` gives, in this order, the streams for
  lengths, K channel scales, q, prefix K, prefix V, suffix K, suffix V, the page
  permutation and the per-step appends.  Large tensors spawn one child stream
  per (head) or (task, head) / (sequence, head) so they can be drawn in
  parallel threads without changing the values.
* Values are drawn in float32 as N(0, 1) times ``value_scale``; K is then
  multiplied per (kv head, channel) by a LogNormal(0, 0.5) factor when
  ``k_channel_scale`` is set; the result is rounded once to bfloat16 with
  round-to-nearest-even.  Arrays hold the bf16 bit patterns as ``uint16``.
* Lengths are integers drawn uniformly with both ends included.
* Suffix slots past a sequence's length, and page slots past the end of a
  sequence's data, hold a bf16 quiet NaN (0x7FC0) so that any read of them
  poisons the result.
"""
from __future__ import annotations

import dataclasses
import math
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, field
from typing import Optional

import numpy as np

BF16_NAN = np.uint16(0x7FC0)

# stream order of SeedSequence(seed).spawn(9)
_S_LEN, _S_KSCALE, _S_Q, _S_PK, _S_PV, _S_SK, _S_SV, _S_PAGES, _S_STEPS = range(9)


def _threads() -> int:
    import os
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (round to nearest, ties to even); return the bit patterns."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    flat = x.reshape(-1)
    out = np.empty(flat.shape, dtype=np.uint16)

    def work(lo: int, hi: int) -> None:
        u = flat[lo:hi].view(np.uint32)
        t = u >> 16
        t &= 1
        t += 0x7FFF
        t += u
        t >>= 16
        out[lo:hi] = t

    n = flat.size
    nt = _threads() if n > (1 << 22) else 1
    step = -(-n // nt) if n else 0
    if nt == 1:
        work(0, n)
    else:
        with ThreadPoolExecutor(nt) as ex:
            list(ex.map(lambda i: work(i * step, min(n, (i + 1) * step)), range(nt)))
    return out.reshape(x.shape)


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns to float32 exactly."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


@dataclass(frozen=True)
class Spec:
    """Shape, value distribution and seed of one synthetic workload."""
    name: str
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    seed: int
    n_branches: int = 5
    prefix_len: int = 0                       # contiguous: shared prefix length
    prefix_range: tuple = (0, 0)              # paged: per-task prefix length range (inclusive)
    suffix_range: tuple = (0, 0)              # per-branch suffix length range (inclusive)
    main_suffix_range: Optional[tuple] = None  # contiguous: sequence 0's own range, drawn after the others
    value_scale: float = 1.0                  # N(0,1) draws are multiplied by this
    k_channel_scale: bool = False             # per-(kv head, channel) LogNormal(0, 0.5) factor on K
    steps: int = 0                            # decode steps with one appended token per branch
    paged: bool = False
    n_tasks: int = 1                          # paged: independent tasks, each with n_branches sequences
    page_size: int = 16
    page_headroom: int = 0                    # paged: extra suffix slots given pre-assigned pages

    @property
    def group(self) -> int:
        return self.n_q_heads // self.n_kv_heads

    @property
    def softmax_scale(self) -> float:
        return 1.0 / math.sqrt(self.head_dim)

    def replace(self, **kw) -> "Spec":
        return dataclasses.replace(self, **kw)


# The five workloads (long agent contexts) and the unscaled Tiny variant.
CONFIGS = {
    "tiny": Spec("tiny", 8, 2, 64, seed=1001, prefix_len=512, suffix_range=(0, 64),
                 value_scale=1.0 / math.sqrt(64)),
    "tiny-unscaled": Spec("tiny-unscaled", 8, 2, 64, seed=1001, prefix_len=512, suffix_range=(0, 64)),
    "mid": Spec("mid", 32, 8, 128, seed=1002, prefix_len=8192, suffix_range=(256, 1024),
                k_channel_scale=True),
    "long": Spec("long", 40, 8, 128, seed=1003, prefix_len=32768, suffix_range=(512, 2048),
                 k_channel_scale=True, steps=256),
    "very-long": Spec("very-long", 64, 8, 128, seed=1004, prefix_len=131072, suffix_range=(1024, 4096),
                      k_channel_scale=True),
    # Fork at turn onset (Sec. 4.4, fork-conditioning comparison): the branches fork before the
    # Thought, so the main sequence's suffix is the whole Thought while the branches' stay short.
    "onset": Spec("onset", 40, 8, 128, seed=1006, prefix_len=32768, suffix_range=(0, 512),
                  main_suffix_range=(4096, 8192), k_channel_scale=True),
    "paged": Spec("paged", 32, 8, 128, seed=1005, paged=True, n_tasks=16, prefix_range=(4096, 65536),
                  suffix_range=(0, 2048), k_channel_scale=True),
}


@dataclass
class ContigWorkload:
    """One decode step (plus optional appends) over a contiguous shared prefix.

    Layouts (bf16 bit patterns, C order):
      q         [N][Hq][d]
      prefix_k  [Hkv][Lp][d]     prefix_v likewise
      suffix_k  [N][Hkv][cap][d] suffix_v likewise; slots >= suffix_len[b] hold NaN
      suffix_len int32 [N]
      step_q    [S][N][Hq][d], step_k / step_v [S][N][Hkv][d]  (appends, in step order)
    """
    spec: Spec
    q: np.ndarray
    prefix_k: np.ndarray
    prefix_v: np.ndarray
    suffix_k: np.ndarray
    suffix_v: np.ndarray
    suffix_len: np.ndarray
    k_scale: Optional[np.ndarray] = None
    step_q: Optional[np.ndarray] = None
    step_k: Optional[np.ndarray] = None
    step_v: Optional[np.ndarray] = None

    @property
    def n_branches(self) -> int:
        return self.q.shape[0]

    @property
    def prefix_len(self) -> int:
        return self.prefix_k.shape[1]

    @property
    def suffix_cap(self) -> int:
        return self.suffix_k.shape[2]


@dataclass
class PagedWorkload:
    """Independent tasks, each a group of sequences sharing its prefix pages.

    Layouts:
      q          [n_seqs][Hq][d] (bf16 bits)
      k_pool     [n_pages][Hkv][page_size][d]   v_pool likewise
      page_table int32 [n_seqs][max_pages]; entry j of sequence i is the pool page holding
                 logical positions [j*P, (j+1)*P).  Positions below the task's prefix length
                 are prefix positions; suffix position u lives at page index ceil(Lp/P) + u//P.
                 Unused entries are -1.
      group_start int32 [n_tasks + 1]; sequences of task t are group_start[t] .. group_start[t+1]-1
      prefix_len  int32 [n_tasks];  suffix_len int32 [n_seqs]; seq_prefix_len int32 [n_seqs]
    """
    spec: Spec
    q: np.ndarray
    k_pool: np.ndarray
    v_pool: np.ndarray
    page_table: np.ndarray
    group_start: np.ndarray
    prefix_len: np.ndarray
    suffix_len: np.ndarray
    suffix_pages: np.ndarray      # pages pre-assigned to each sequence's suffix
    k_scale: Optional[np.ndarray] = None

    @property
    def n_seqs(self) -> int:
        return self.q.shape[0]

    @property
    def seq_prefix_len(self) -> np.ndarray:
        out = np.empty(self.n_seqs, np.int32)
        for t in range(len(self.prefix_len)):
            out[self.group_start[t]:self.group_start[t + 1]] = self.prefix_len[t]
        return out


def _normal(ss: np.random.SeedSequence, shape, scale: float) -> np.ndarray:
    g = np.random.Generator(np.random.PCG64(ss))
    x = g.standard_normal(shape, dtype=np.float32)
    if scale != 1.0:
        x *= np.float32(scale)
    return x


def _kv_block(ss: np.random.SeedSequence, shape, spec: Spec, kscale_row: Optional[np.ndarray]) -> np.ndarray:
    """Draw one [..., d] block, apply the K channel scale if given, round to bf16."""
    x = _normal(ss, shape, spec.value_scale)
    if kscale_row is not None:
        x *= kscale_row
    return bf16_bits(x)


def _draw_kscale(ss: np.random.SeedSequence, spec: Spec) -> Optional[np.ndarray]:
    if not spec.k_channel_scale:
        return None
    g = np.random.Generator(np.random.PCG64(ss))
    return g.lognormal(0.0, 0.5, size=(spec.n_kv_heads, spec.head_dim)).astype(np.float32)


def make_contig(spec: Spec) -> ContigWorkload:
    """Materialise a contiguous-KV workload from its spec (deterministic in spec.seed)."""
    assert not spec.paged
    N, Hq, Hkv, d = spec.n_branches, spec.n_q_heads, spec.n_kv_heads, spec.head_dim
    streams = np.random.SeedSequence(spec.seed).spawn(9)
    lens_rng = np.random.Generator(np.random.PCG64(streams[_S_LEN]))
    lo, hi = spec.suffix_range
    suffix_len = lens_rng.integers(lo, hi, size=N, endpoint=True).astype(np.int32)
    if spec.main_suffix_range is not None:
        mlo, mhi = spec.main_suffix_range
        suffix_len[0] = lens_rng.integers(mlo, mhi, endpoint=True)
        hi = max(hi, mhi)
    cap = max(1, hi + spec.steps)
    kscale = _draw_kscale(streams[_S_KSCALE], spec)

    q = bf16_bits(_normal(streams[_S_Q], (N, Hq, d), spec.value_scale))
    Lp = spec.prefix_len
    prefix_k = np.empty((Hkv, Lp, d), np.uint16)
    prefix_v = np.empty((Hkv, Lp, d), np.uint16)
    suffix_k = np.full((N, Hkv, cap, d), BF16_NAN, np.uint16)
    suffix_v = np.full((N, Hkv, cap, d), BF16_NAN, np.uint16)
    pk_ss = streams[_S_PK].spawn(Hkv)
    pv_ss = streams[_S_PV].spawn(Hkv)
    sk_ss = streams[_S_SK].spawn(N * Hkv)
    sv_ss = streams[_S_SV].spawn(N * Hkv)

    jobs = []
    for g in range(Hkv):
        ks = None if kscale is None else kscale[g]
        jobs.append((prefix_k, (g,), pk_ss[g], (Lp, d), ks))
        jobs.append((prefix_v, (g,), pv_ss[g], (Lp, d), None))
    for b in range(N):
        L = int(suffix_len[b])
        for g in range(Hkv):
            ks = None if kscale is None else kscale[g]
            jobs.append((suffix_k, (b, g, slice(0, L)), sk_ss[b * Hkv + g], (L, d), ks))
            jobs.append((suffix_v, (b, g, slice(0, L)), sv_ss[b * Hkv + g], (L, d), None))

    def run(job):
        dst, idx, ss, shape, ks = job
        dst[idx] = _kv_block(ss, shape, spec, ks)

    with ThreadPoolExecutor(_threads()) as ex:
        list(ex.map(run, jobs))

    step_q = step_k = step_v = None
    if spec.steps:
        g = np.random.Generator(np.random.PCG64(streams[_S_STEPS]))
        sq, sk, sv = [], [], []
        for _ in range(spec.steps):
            qs = g.standard_normal((N, Hq, d), dtype=np.float32) * np.float32(spec.value_scale)
            k = g.standard_normal((N, Hkv, d), dtype=np.float32) * np.float32(spec.value_scale)
            v = g.standard_normal((N, Hkv, d), dtype=np.float32) * np.float32(spec.value_scale)
            if kscale is not None:
                k *= kscale[None]
            sq.append(qs), sk.append(k), sv.append(v)
        step_q = bf16_bits(np.stack(sq))
        step_k = bf16_bits(np.stack(sk))
        step_v = bf16_bits(np.stack(sv))
    return ContigWorkload(spec, q, prefix_k, prefix_v, suffix_k, suffix_v, suffix_len, kscale,
                          step_q, step_k, step_v)


def make_paged(spec: Spec) -> PagedWorkload:
    """Materialise a paged workload: tasks x branches sequences over a permuted page pool."""
    assert spec.paged
    T, B, Hq, Hkv, d, P = spec.n_tasks, spec.n_branches, spec.n_q_heads, spec.n_kv_heads, spec.head_dim, spec.page_size
    S = T * B
    streams = np.random.SeedSequence(spec.seed).spawn(9)
    lens_rng = np.random.Generator(np.random.PCG64(streams[_S_LEN]))
    plo, phi = spec.prefix_range
    prefix_len = lens_rng.integers(plo, phi, size=T, endpoint=True).astype(np.int32)
    slo, shi = spec.suffix_range
    suffix_len = lens_rng.integers(slo, shi, size=S, endpoint=True).astype(np.int32)
    kscale = _draw_kscale(streams[_S_KSCALE], spec)
    q = bf16_bits(_normal(streams[_S_Q], (S, Hq, d), spec.value_scale))
    group_start = (np.arange(T + 1, dtype=np.int32) * B).astype(np.int32)

    # logical page order: task-major, the task's prefix pages, then each branch's suffix pages
    n_pre = [-(-int(L) // P) for L in prefix_len]
    n_suf = [-(-(int(L) + spec.page_headroom) // P) for L in suffix_len]
    n_pages = sum(n_pre) + sum(n_suf)
    perm = np.random.Generator(np.random.PCG64(streams[_S_PAGES])).permutation(n_pages).astype(np.int32)
    # wide enough for any task's prefix plus the longest suffix (plus headroom) of any sequence
    max_pages = max(n_pre) + max(n_suf)
    page_table = np.full((S, max(1, max_pages)), -1, np.int32)
    suffix_pages = np.full((S, max(1, max(n_suf) if n_suf else 1)), -1, np.int32)
    cursor = 0
    prefix_pages = []
    for t in range(T):
        pp = perm[cursor:cursor + n_pre[t]]
        cursor += n_pre[t]
        prefix_pages.append(pp)
        for b in range(B):
            i = t * B + b
            sp = perm[cursor:cursor + n_suf[i]]
            cursor += n_suf[i]
            page_table[i, :n_pre[t]] = pp
            page_table[i, n_pre[t]:n_pre[t] + n_suf[i]] = sp
            suffix_pages[i, :n_suf[i]] = sp
    assert cursor == n_pages

    k_pool = np.full((n_pages, Hkv, P, d), BF16_NAN, np.uint16)
    v_pool = np.full((n_pages, Hkv, P, d), BF16_NAN, np.uint16)
    pk_ss = streams[_S_PK].spawn(T * Hkv)
    pv_ss = streams[_S_PV].spawn(T * Hkv)
    sk_ss = streams[_S_SK].spawn(S * Hkv)
    sv_ss = streams[_S_SV].spawn(S * Hkv)

    def scatter(pool, pages, g, block):
        L = block.shape[0]
        full = L // P
        if full:
            pool[pages[:full], g] = block[:full * P].reshape(full, P, d)
        rem = L - full * P
        if rem:
            pool[pages[full], g, :rem] = block[full * P:]

    jobs = []
    for t in range(T):
        for g in range(Hkv):
            ks = None if kscale is None else kscale[g]
            jobs.append((k_pool, prefix_pages[t], g, pk_ss[t * Hkv + g], int(prefix_len[t]), ks))
            jobs.append((v_pool, prefix_pages[t], g, pv_ss[t * Hkv + g], int(prefix_len[t]), None))
    for i in range(S):
        for g in range(Hkv):
            ks = None if kscale is None else kscale[g]
            jobs.append((k_pool, suffix_pages[i], g, sk_ss[i * Hkv + g], int(suffix_len[i]), ks))
            jobs.append((v_pool, suffix_pages[i], g, sv_ss[i * Hkv + g], int(suffix_len[i]), None))

    def run(job):
        pool, pages, g, ss, L, ks = job
        scatter(pool, pages, g, _kv_block(ss, (L, d), spec, ks))

    # distinct jobs write distinct (page, head) blocks, so threads never overlap
    with ThreadPoolExecutor(_threads()) as ex:
        list(ex.map(run, jobs))
    return PagedWorkload(spec, q, k_pool, v_pool, page_table, group_start, prefix_len, suffix_len,
                         suffix_pages, kscale)


def make(name_or_spec, **overrides):
    """Build the named workload (``CONFIGS`` key) or an explicit Spec, with optional field overrides."""
    spec = CONFIGS[name_or_spec] if isinstance(name_or_spec, str) else name_or_spec
    if overrides:
        spec = spec.replace(**overrides)
    return make_paged(spec) if spec.paged else make_contig(spec)


def kv_bytes_contig(w: ContigWorkload, suffix_len: Optional[np.ndarray] = None) -> dict:
    """Algorithmic K+V bytes of one decode step: the prefix once plus every branch's own suffix."""
    sl = w.suffix_len if suffix_len is None else suffix_len
    per_tok = 2 * w.spec.n_kv_heads * w.spec.head_dim * 2
    pre = w.prefix_len * per_tok
    suf = int(np.sum(sl)) * per_tok
    naive = w.n_branches * pre + suf
    return {"prefix": pre, "suffix": suf, "total": pre + suf, "naive": naive}


def kv_bytes_paged(w: PagedWorkload) -> dict:
    per_tok = 2 * w.spec.n_kv_heads * w.spec.head_dim * 2
    pre = int(np.sum(w.prefix_len)) * per_tok
    suf = int(np.sum(w.suffix_len)) * per_tok
    naive = sum(int(w.prefix_len[t]) * (int(w.group_start[t + 1]) - int(w.group_start[t]))
                for t in range(len(w.prefix_len))) * per_tok + suf
    return {"prefix": pre, "suffix": suf, "total": pre + suf, "naive": naive}
