"""Fork-aware decode attention benchmark (one GPU).

A step is one fork-decode step of one attention layer: every sequence of the fork
(main thread + 4 branches) appends its new K/V token and attends with one new query
over the shared prefix and its own suffix.  The default workload is the long agent
context: 32768-token shared prefix, 5 sequences, 40 query / 8 KV heads, head_dim 128,
suffixes of 512..2048 tokens, 256 appended tokens per layer.  Layers are replicated
so that the working set (>= 1 GiB) exceeds the 256 MB Infinity Cache and every step
reads HBM; step i runs on replica i % R.  Inputs are resident in HBM before the timed
region.  The timed region is K steps launched as one HIP graph (captured once, so host
launch overhead is not measured); it runs in several trials, each from the same suffix
lengths, and the median trial is reported.  The same JSON line carries sub-records for
the other workloads (128k prefix, 16 paged forks, 8k prefix), each timed the same way,
a read-only bandwidth probe and the CPU oracle's rate.  Prints one JSON line.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBPS = 8000.0
MALL_BYTES = 256 << 20
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")
KERNEL_SOURCE = os.path.join(ROOT, "paper_2608_13667_amd", "csrc", "partials.hip")
SUB_WORKLOADS = ("very-long", "paged", "mid", "onset", "tiny")


def measured_traffic(workload: str):
    """HBM bytes per launch of the partial-attention kernel from the committed counter
    summary, or None when it was taken on another workload or another kernel source."""
    import hashlib
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
        with open(KERNEL_SOURCE, "rb") as f:
            digest = hashlib.sha256(f.read()).hexdigest()
    except (OSError, ValueError):
        return None
    entry = rec.get(workload)
    if not entry or entry.get("kernel_sha256") != digest:
        return None
    return entry.get("bytes_per_launch")


DESCRIPTIONS = {
    "long": "long agent context: 32768-token shared prefix, 5 sequences (main + 4 branches), 40 q / 8 kv heads, "
            "head_dim 128, suffixes 512..2048 tokens, one appended token per sequence per step",
    "very-long": "very long context: 131072-token shared prefix, 5 sequences, 64 q / 8 kv heads, head_dim 128, "
                 "suffixes 1024..4096 tokens",
    "mid": "mid context: 8192-token shared prefix, 5 sequences, 32 q / 8 kv heads, head_dim 128, "
           "suffixes 256..1024 tokens",
    "tiny": "tiny: 512-token shared prefix, 5 sequences, 8 q / 2 kv heads, head_dim 64, suffixes 0..64 tokens",
    "onset": "fork at turn onset: 32768-token shared prefix, 5 sequences, 40 q / 8 kv heads, head_dim 128, "
             "main suffix 4096..8192 tokens (the Thought), branch suffixes 0..512",
    "paged": "concurrent agents, paged: 16 tasks x 5 sequences, 32 q / 8 kv heads, head_dim 128, prefixes "
             "4096..65536, suffixes 0..2048, 16-token pages from a permuted pool",
}


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None,
                    help="timed steps per trial (default: 256 appends per replica for the long workload)")
    ap.add_argument("--warmup", type=int, default=20, help="untimed steps before the timed trials")
    ap.add_argument("--trials", type=int, default=5, help="timed trials; the median is reported")
    ap.add_argument("--workload", default="long", choices=sorted(DESCRIPTIONS))
    ap.add_argument("--sub", default=",".join(SUB_WORKLOADS),
                    help="comma-separated workloads timed as sub-records ('' for none)")
    ap.add_argument("--replicas", type=int, default=0, help="layer replicas (0: enough for >= 1 GiB)")
    ap.add_argument("--rounds", type=int, default=0, help="schedule rounds of the resident waves (0: automatic)")
    ap.add_argument("--eager", action="store_true", help="launch the timed steps one by one instead of as a graph")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-naive", action="store_true", help="skip the naive per-branch GPU baseline")
    ap.add_argument("--no-probe", action="store_true", help="skip the read-bandwidth probe")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-prefill", action="store_true", help="skip the instruction-prefill timing")
    ap.add_argument("--yardstick-copy", action="store_true",
                    help="first copy 256 MiB device to device (a kernel of known traffic, to scale HBM counters)")
    ap.add_argument("--prefill-only", action="store_true",
                    help="time only the instruction prefill (for profiling its kernel alone)")
    ap.add_argument("--prefill-tokens", default="1,16,64", help="instruction tokens per branch to time")
    ap.add_argument("--lifecycle", action="store_true",
                    help="also time the fork lifecycle on the page pool (contiguous workloads' shapes)")
    return ap.parse_args()


class Bench:
    """One workload on the device: layer replicas, plans, step and partial-kernel timing."""

    def __init__(self, torch, fa, W, name, args):
        self.torch, self.fa, self.W, self.name, self.args = torch, fa, W, name, args
        t0 = time.time()
        w = self.w = W.make(name)
        log(f"[bench] generated {name} in {time.time() - t0:.1f}s")
        spec = self.spec = w.spec
        self.paged = spec.paged
        self.appends = spec.steps > 0
        self.kvb = W.kv_bytes_paged(w) if self.paged else W.kv_bytes_contig(w)
        self.R = args.replicas or max(1, math.ceil((1 << 30) / self.kvb["total"]))
        dev = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
        if self.paged:
            base = dict(q=dev(w.q), k_pool=dev(w.k_pool), v_pool=dev(w.v_pool),
                        page_table=torch.from_numpy(w.page_table).cuda(),
                        suffix_len=torch.from_numpy(w.suffix_len).cuda())
        else:
            base = dict(q=dev(w.q), prefix_k=dev(w.prefix_k), prefix_v=dev(w.prefix_v), suffix_k=dev(w.suffix_k),
                        suffix_v=dev(w.suffix_v), suffix_len=torch.from_numpy(w.suffix_len).cuda())
        self.reps = [base] + [{k: v.clone() for k, v in base.items()} for _ in range(self.R - 1)]
        self.n_seq = w.q.shape[0]
        self.out = torch.empty((self.n_seq, spec.n_q_heads, spec.head_dim), device="cuda")
        self.lse = torch.empty((self.n_seq, spec.n_q_heads), device="cuda")
        if self.appends:
            self.step_q, self.step_k, self.step_v = dev(w.step_q), dev(w.step_k), dev(w.step_v)
        self.len0 = torch.from_numpy(w.suffix_len).cuda()
        self.per_tok = 2 * spec.n_kv_heads * spec.head_dim * 2
        log(f"[bench] {name}: {self.R} replicas x {self.kvb['total'] / 2**20:.1f} MiB")

    def default_steps(self):
        return 256 * self.R if self.appends else max(200, 20 * self.R)

    def plan(self, share=True):
        spec, w, fa = self.spec, self.w, self.fa
        if self.paged:
            return fa.Plan.paged_plan(spec.n_q_heads, spec.n_kv_heads, spec.head_dim, w.group_start, w.prefix_len,
                                      w.page_table.shape[1], w.k_pool.shape[0], int(w.suffix_len.max()),
                                      share_prefix=share, rounds=self.args.rounds)
        return fa.Plan.contig(spec.n_q_heads, spec.n_kv_heads, spec.head_dim, w.n_branches, w.prefix_len,
                              w.suffix_cap, w.suffix_cap, share_prefix=share, rounds=self.args.rounds)

    def run(self, plan, i):
        r = self.reps[i % self.R]
        if self.paged:
            plan.decode_paged(r["q"], r["k_pool"], r["v_pool"], r["page_table"], r["suffix_len"], self.out, self.lse)
        elif self.appends:
            j = i // self.R
            plan.step(self.step_q[j], self.step_k[j], self.step_v[j], r["prefix_k"], r["prefix_v"], r["suffix_k"],
                      r["suffix_v"], r["suffix_len"], self.out, self.lse)
        else:
            plan.decode(r["q"], r["prefix_k"], r["prefix_v"], r["suffix_k"], r["suffix_v"], r["suffix_len"], self.out,
                        self.lse)

    def reset(self):
        for r in self.reps:
            r["suffix_len"].copy_(self.len0)

    def timed(self, body, n, warmup_body=None, trials=5):
        """Seconds of each trial of body(n).  With graphs, the n calls are captured once and each
        trial replays them; the suffix lengths are reset before every trial (outside the timing)."""
        torch = self.torch
        if warmup_body is not None:
            warmup_body()
        torch.cuda.synchronize()
        graph = None
        if not self.args.eager:
            self.reset()
            torch.cuda.synchronize()
            graph = torch.cuda.CUDAGraph()
            with torch.cuda.graph(graph):
                body(n)
            torch.cuda.synchronize()
        out = []
        for _ in range(trials):
            self.reset()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            if graph is not None:
                graph.replay()
            else:
                body(n)
            e1.record()
            torch.cuda.synchronize()
            out.append(e0.elapsed_time(e1) * 1e-3)
        return out

    def step_bytes(self, n_steps):
        """Algorithmic K/V bytes of n steps: each group's prefix once per step plus every suffix at its length."""
        total = 0
        sl0 = int(np.sum(self.w.suffix_len))
        for i in range(n_steps):
            extra = (i // self.R + 1) * self.n_seq if self.appends else 0
            total += self.kvb["prefix"] + (sl0 + extra) * self.per_tok
        return total

    def partial_kernel(self, plan, step_s):
        """Average duration of the partial-attention kernel alone (its launches replayed as one graph on
        the stream they run on), as the suffix lengths of the first step leave it.  step_s: the
        measured step time, which sizes the trials."""
        torch = self.torch
        info = plan.info()
        d = self.spec.head_dim
        po = torch.empty((info.n_slots, info.slot_rows, d), device="cuda")
        pl = torch.empty((info.n_slots, info.slot_rows), device="cuda")

        def part(n):
            for i in range(n):
                r = self.reps[i % self.R]
                if self.paged:
                    plan.partials_paged(r["q"], r["k_pool"], r["v_pool"], r["page_table"], r["suffix_len"], po, pl)
                else:
                    plan.partials(r["q"], r["prefix_k"], r["prefix_v"], r["suffix_k"], r["suffix_v"], r["suffix_len"],
                                  po, pl)
        # at least 60 launches and about 20 ms of them per trial, and the median of 5 trials: the
        # device's clock settles over a few milliseconds of back-to-back launches (20 launches of the
        # 128k workload, or 200 of the tiny one, do not span that)
        kp = max(60, min(4000, int(0.02 / max(step_s, 1e-6))))
        secs = self.timed(part, kp, warmup_body=lambda: part(10), trials=5)
        return float(np.median(secs)) / kp

    def measure(self, n_steps, warmup, trials, naive=True, mall_warm=False):
        """Fork-aware steps (median of trials), the partial kernel alone, the naive baseline."""
        plan = self.plan(True)
        info = plan.info()
        secs = self.timed(lambda n: [self.run(plan, i) for i in range(n)], n_steps,
                          warmup_body=lambda: [self.run(plan, i) for i in range(warmup)], trials=trials)
        assert plan.device_error() == 0, "device error flag raised"
        med = float(np.median(secs))
        alg = self.step_bytes(n_steps)
        gbps = alg / med / 1e9
        k_secs = self.partial_kernel(plan, med / n_steps)
        k_gbps = self.kvb["total"] / k_secs / 1e9
        rec = {"steps_per_s": n_steps / med, "us_per_step": med / n_steps * 1e6,
               "trials_us_per_step": [s / n_steps * 1e6 for s in secs], "steps": n_steps, "warmup": warmup,
               "effective_kv_gbps": gbps, "hbm_peak_frac": gbps / HBM_PEAK_GBPS,
               "roofline": {"bound": "hbm", "kernel": "partials_kernel (prefix + suffix partial attention)",
                            "achieved": k_gbps, "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": k_gbps / HBM_PEAK_GBPS,
                            "traffic": measured_traffic(self.name), "avg_launch_us": k_secs * 1e6,
                            "bytes_per_launch": self.kvb["total"]},
               "config": {"workload": DESCRIPTIONS[self.name], "name": self.name, "replicas": self.R,
                          "working_set_gib": self.R * self.kvb["total"] / 2**30, "blocks": info.n_blocks,
                          "waves_per_block": info.waves_per_block, "rounds": info.rounds, "work_items": info.n_items,
                          "static_split": bool(info.static_split),
                          "launch": "eager" if self.args.eager else "hip graph of the timed steps"}}
        log(f"[bench] {self.name} fork-aware: {rec['steps_per_s']:.1f} steps/s, {rec['us_per_step']:.2f} us/step, "
            f"{gbps:.0f} GB/s ({rec['hbm_peak_frac'] * 100:.1f}% of 8 TB/s); partial kernel {k_secs * 1e6:.2f} us, "
            f"{k_gbps / HBM_PEAK_GBPS * 100:.1f}%")
        if naive:
            nplan = self.plan(False)
            kn = max(self.R, n_steps // 4)
            nsecs = self.timed(lambda n: [self.run(nplan, i) for i in range(n)], kn,
                               warmup_body=lambda: [self.run(nplan, i) for i in range(min(warmup, kn))], trials=3)
            nmed = float(np.median(nsecs))
            nalg = self.step_bytes(kn)
            rec["naive_per_branch"] = {
                "steps_per_s": kn / nmed, "us_per_step": nmed / kn * 1e6, "effective_kv_gbps": nalg / nmed / 1e9,
                "requested_kv_gbps": (nalg + (self.kvb["naive"] - self.kvb["total"]) * kn) / nmed / 1e9,
                "prefix_reuse_speedup": (nmed / kn) / (med / n_steps)}
            log(f"[bench] {self.name} naive: {kn / nmed:.1f} steps/s, speed-up of sharing "
                f"{rec['naive_per_branch']['prefix_reuse_speedup']:.2f}x")
            nplan.close()
        if mall_warm and not self.paged and self.kvb["total"] < MALL_BYTES:
            r0 = self.reps[0]
            nw = min(n_steps, 200)
            ws = self.timed(lambda n: [plan.decode(r0["q"], r0["prefix_k"], r0["prefix_v"], r0["suffix_k"],
                                                   r0["suffix_v"], r0["suffix_len"], self.out, self.lse)
                                       for _ in range(n)], nw, trials=3)
            wmed = float(np.median(ws))
            rec["mall_warm_single_replica"] = {"steps_per_s": nw / wmed, "kv_gbps": self.kvb["total"] * nw / wmed / 1e9}
        self.plan_info = info
        plan.close()
        return rec

    def release(self):
        self.reps = None
        self.torch.cuda.empty_cache()


def read_probe(torch, fa, sizes):
    """Achievable read bandwidth: the library's streaming read kernel over buffers rotated so that
    >= 1 GiB is touched between repeats of one buffer, for a few launch shapes; the best is kept."""
    sink = torch.zeros(64, dtype=torch.int32, device="cuda")
    out = {}
    for label, nbytes in sizes.items():
        nbytes = nbytes // 4096 * 4096
        R = max(2, math.ceil((1 << 30) / nbytes))
        bufs = [torch.empty(nbytes // 4, dtype=torch.int32, device="cuda").fill_(i) for i in range(R)]
        best = None
        for blocks, threads, unroll in ((4096, 512, 4), (2048, 256, 8), (1024, 512, 8), (256, 512, 4)):
            def go(n):
                for i in range(n):
                    fa.read_probe(bufs[i % R], blocks, threads, unroll, sink)
            go(4)
            torch.cuda.synchronize()
            n = max(20, 2 * R)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            go(n)
            e1.record()
            torch.cuda.synchronize()
            us = e0.elapsed_time(e1) * 1e3 / n
            g = nbytes / us / 1e3
            if best is None or g > best["gbps"]:
                best = {"gbps": g, "us": us, "bytes": nbytes, "blocks": blocks, "threads": threads, "unroll": unroll}
        out[label] = best
        del bufs
        torch.cuda.empty_cache()
        log(f"[bench] read probe {label}: {best['gbps']:.0f} GB/s ({best['us']:.2f} us for {nbytes / 2**20:.1f} MiB)")
    return out


def cpu_oracle(oracle, w, n_seq, hq, seconds):
    """The fp64 oracle on the host: all rows of full decode steps at the initial lengths, on every
    host thread and on one."""
    oracle.build(force=False)
    res = {}
    for label, threads in (("all", None), ("one", 1)):
        if threads is not None:
            oracle.set_threads(threads)
        n, t0 = 0, time.time()
        budget = seconds if threads is None else seconds / 2
        while True:
            oracle.decode_workload(w)
            n += 1
            if time.time() - t0 >= budget:
                break
        res[label] = (n / (time.time() - t0), oracle.threads(), n)
    oracle.set_threads(len(os.sched_getaffinity(0)))
    v, cores, n = res["all"]
    v1, _, n1 = res["one"]
    log(f"[bench] cpu oracle: {v:.3f} steps/s on {cores} threads, {v1:.4f} steps/s on 1")
    return {"value": v, "unit": "steps/s", "cores": cores, "kind": "oracle",
            "sample": f"{n} full decode steps (all {n_seq} x {hq} rows) at the initial lengths, fp64 on the host",
            "single_thread": {"value": v1, "unit": "steps/s", "cores": 1, "sample": f"{n1} full decode steps"}}


def lifecycle_timing(fa, torch, w):
    """One turn transition of the fork lifecycle at the workload's shape, with a page pool: fork
    the snapshot to all sequences, reserve their suffix pages, drop the branches, promote the main
    sequence (host bookkeeping), the promote's device work (a gather of the main context's tail,
    from the first page the dense layout rewrites, and its scatter into the dense pages), and the
    branches' instruction prefill on the pool after a fork (fka_prefill_paged, 16 tokens per
    branch) and the harvest's prefill of 256 tokens into the promoted main context.  Host calls are timed with perf_counter over many cycles, the device work with HIP
    events on the launch stream."""
    spec = w.spec
    N, Hkv, d = w.n_branches, spec.n_kv_heads, spec.head_dim
    Lp, lens = w.prefix_len, [int(x) for x in w.suffix_len]
    a = -(-Lp // 16)
    max_pages = a + -(-max(lens) // 16) + 1
    n_pages = a + sum(-(-L // 16) for L in lens) + -(-(Lp + max(lens)) // 16) + 8
    pool = fa.Pool(n_pages)
    pages = torch.zeros((n_pages, Hkv, 16, d), dtype=torch.bfloat16, device="cuda")
    v_pages = torch.zeros_like(pages)
    host = {"fork": [], "reserve": [], "drop": [], "promote": []}
    cycles = 50
    for _ in range(cycles):
        snap = pool.alloc(a)
        table = np.full((N, max_pages), -1, np.int32)
        t0 = time.perf_counter()
        pool.fork(snap, table, 0, N)
        t1 = time.perf_counter()
        for b in range(N):
            pool.reserve(table, b, Lp, lens[b])
        t2 = time.perf_counter()
        for b in range(1, N):
            pool.drop(table, b)
        t3 = time.perf_counter()
        dense, frm = pool.promote(table, 0, Lp, lens[0])
        t4 = time.perf_counter()
        host["fork"].append(t1 - t0)
        host["reserve"].append((t2 - t1) / N)
        host["drop"].append((t3 - t2) / (N - 1))
        host["promote"].append(t4 - t3)
        pool.release(snap)
        pool.release(dense)
    assert pool.free_pages() == n_pages
    # device work of one promote, on a table from a fresh fork
    snap = pool.alloc(a)
    table = np.full((N, max_pages), -1, np.int32)
    pool.fork(snap, table, 0, N)
    pool.reserve(table, 0, Lp, lens[0])
    L0 = Lp + lens[0]
    plan = fa.Plan.paged_plan(spec.n_q_heads, Hkv, d, [0, N], [Lp], max_pages, n_pages, max(lens))
    old_row = torch.from_numpy(table).cuda()
    for b in range(1, N):
        pool.drop(table, b)
    dense, frm = pool.promote(table, 0, Lp, lens[0])
    dense_dev = torch.from_numpy(dense).cuda()
    tmp_k = torch.empty((Hkv, L0 - frm, d), dtype=torch.bfloat16, device="cuda")
    tmp_v = torch.empty_like(tmp_k)
    stream = torch.cuda.current_stream()

    def promote_device():
        plan.gather_paged_range(0, frm, L0, pages, v_pages, old_row, tmp_k, tmp_v, stream)
        fa.scatter_pages(tmp_k, tmp_v, frm, dense_dev, n_pages, pages, v_pages, None, stream)

    for _ in range(5):
        promote_device()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    reps = 20
    e0.record(stream)
    for _ in range(reps):
        promote_device()
    e1.record(stream)
    torch.cuda.synchronize()
    dev_s = e0.elapsed_time(e1) / 1e3 / reps
    per_tok = Hkv * d * 2 * 2
    moved = 4 * per_tok * (L0 - frm)  # the gather and the scatter each read and write L0 - frm tokens
    plan.close()
    pool.release(dense)
    pool.release(snap)
    # branch-instruction prefill on the pool (fka_prefill_paged): after a fresh fork (empty
    # suffixes) every branch takes n instruction tokens into pages reserved for them (MALL-warm:
    # one pool)
    n = 16
    Hq = spec.n_q_heads
    table = np.full((N, max_pages), -1, np.int32)
    snap2 = pool.alloc(a)
    pool.fork(snap2, table, 0, N)
    for b in range(N):
        pool.reserve(table, b, Lp, n)
    pplan = fa.Plan.prefill_paged_plan(Hq, Hkv, d, N, n, Lp, max_pages, n_pages, n)
    vt = torch.from_numpy(table).cuda()
    lens_dev = torch.zeros(N, dtype=torch.int32, device="cuda")
    q = torch.zeros((N, n, Hq, d), dtype=torch.bfloat16, device="cuda")
    o = torch.empty((N, n, Hq, d), device="cuda")
    for _ in range(5):
        pplan.prefill_paged(q, pages, v_pages, vt, lens_dev, o, None, stream)
    e0.record(stream)
    for _ in range(reps):
        pplan.prefill_paged(q, pages, v_pages, vt, lens_dev, o, None, stream)
    e1.record(stream)
    torch.cuda.synchronize()
    pf_s = e0.elapsed_time(e1) / 1e3 / reps
    # the prefix once, each branch's instruction
    pf_bytes = per_tok * (Lp + N * n)
    # thought harvesting: the promoted main context takes h harvested tokens (one sequence)
    h = 256
    mp2 = -(-L0 // 16) + -(-h // 16)
    snap3 = pool.alloc(-(-L0 // 16))
    t3 = np.full((1, mp2), -1, np.int32)
    pool.fork(snap3, t3, 0, 1)
    pool.reserve(t3, 0, L0, h)
    hplan = fa.Plan.prefill_paged_plan(Hq, Hkv, d, 1, h, L0, mp2, n_pages, h)
    t3d = torch.from_numpy(t3).cuda()
    len1 = torch.zeros(1, dtype=torch.int32, device="cuda")
    qh = torch.zeros((1, h, Hq, d), dtype=torch.bfloat16, device="cuda")
    oh = torch.empty((1, h, Hq, d), device="cuda")
    for _ in range(5):
        hplan.prefill_paged(qh, pages, v_pages, t3d, len1, oh, None, stream)
    e0.record(stream)
    for _ in range(reps):
        hplan.prefill_paged(qh, pages, v_pages, t3d, len1, oh, None, stream)
    e1.record(stream)
    torch.cuda.synchronize()
    hv_s = e0.elapsed_time(e1) / 1e3 / reps
    hplan.close()
    pplan.close()
    pool.close()
    ms = lambda v: float(np.median(v) * 1e6)
    return {"tokens_promoted": L0, "host_us": {k: ms(v) for k, v in host.items()},
            "promote_device_us": dev_s * 1e6, "promote_device_gbps": moved / dev_s / 1e9,
            "prefill_paged": {"tokens_per_branch": n, "us": pf_s * 1e6, "us_per_token": pf_s * 1e6 / (N * n),
                              "kv_gbps": pf_bytes / pf_s / 1e9, "cache": "MALL-warm (one pool)"},
            "harvest_prefill_paged": {"tokens": h, "context": L0, "us": hv_s * 1e6, "us_per_token": hv_s * 1e6 / h,
                                      "cache": "MALL-warm (one pool)"}}


def prefill_timing(torch, fa, W, ns, trials):
    """Instruction prefill at the 32k-prefix shape (fka_prefill): every branch takes n instruction
    tokens at the fork (existing suffixes empty).  HBM-cold: the calls cycle over prefix replicas
    totalling 3x the 256 MiB MALL.  Per n: us per call and per token, effective K/V GB/s (the
    prefix once, each branch's instruction once) against 8 TB/s, and MFMA TFLOP/s (4 Lp d per
    query row: q.k and p.v over the prefix) against the 2.5 PFLOP/s bf16 peak; and the same calls
    over a page pool with permuted page ids (fka_prefill_paged)."""
    n_max = max(ns)
    w = W.make("long", steps=n_max, suffix_range=(0, 0), seed=2700)
    s = w.spec
    N, Hq, Hkv, d, Lp = w.q.shape[0], s.n_q_heads, s.n_kv_heads, s.head_dim, w.prefix_len
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
    sk, sv = w.suffix_k.copy(), w.suffix_v.copy()
    for b in range(N):
        sk[b, :, :n_max] = w.step_k[:n_max, b].transpose(1, 0, 2)
        sv[b, :, :n_max] = w.step_v[:n_max, b].transpose(1, 0, 2)
    q_all = w.step_q.transpose(1, 0, 2, 3)
    pref_bytes = 2 * Hkv * Lp * d * 2
    R = max(2, math.ceil(3 * 256 * 2**20 / pref_bytes))
    pk0, pv0 = dev(w.prefix_k), dev(w.prefix_v)
    reps = [(pk0, pv0)] + [(pk0.clone(), pv0.clone()) for _ in range(R - 1)]
    skd, svd = dev(sk), dev(sv)
    len0 = torch.zeros(N, dtype=torch.int32, device="cuda")
    cap = w.suffix_cap
    # the same K/V in a page pool (fka_prefill_paged): 16-token pages whose ids are a seeded
    # permutation, the prefix pages shared by every branch's row; R pool replicas, as above
    npre, nsuf = -(-Lp // 16), -(-cap // 16)
    perm = np.random.default_rng(2701).permutation(npre + N * nsuf)
    table = np.empty((N, npre + nsuf), np.int32)
    pools = []
    for src_p, src_s in ((w.prefix_k, sk), (w.prefix_v, sv)):
        pool = np.zeros((npre + N * nsuf, Hkv, 16, d), np.uint16)
        pad = np.zeros((Hkv, npre * 16, d), np.uint16)
        pad[:, :Lp] = src_p
        pool[perm[:npre]] = pad.reshape(Hkv, npre, 16, d).transpose(1, 0, 2, 3)
        for b in range(N):
            spad = np.zeros((Hkv, nsuf * 16, d), np.uint16)
            spad[:, :cap] = src_s[b]
            ids = perm[npre + b * nsuf:npre + (b + 1) * nsuf]
            pool[ids] = spad.reshape(Hkv, nsuf, 16, d).transpose(1, 0, 2, 3)
            table[b] = np.concatenate([perm[:npre], ids])
        pools.append(pool)
    kp0, vp0 = dev(pools[0]), dev(pools[1])
    del pools
    preps = [(kp0, vp0)] + [(kp0.clone(), vp0.clone()) for _ in range(R - 1)]
    tab = torch.from_numpy(table).cuda()
    res = {"workload": "long: 40 query / 8 KV heads, d 128, 32768-token prefix, 5 branches, empty suffixes",
           "replicas": R, "cold": "calls cycle over prefix replicas of 3x the MALL",
           "paged": "the same calls over a page pool with permuted page ids (fka_prefill_paged)"}

    def timed(call):
        K = 4 * R
        for i in range(2 * R):
            call(i)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph):
            for i in range(K):
                call(i)
        torch.cuda.synchronize()
        ts = []
        for _ in range(trials):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            graph.replay()
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1) * 1e-3 / K)
        del graph
        return float(np.median(ts)), ts

    for n in ns:
        plan = fa.Plan.prefill_plan(Hq, Hkv, d, N, n, Lp, cap, cap)
        pplan = fa.Plan.prefill_paged_plan(Hq, Hkv, d, N, n, Lp, table.shape[1], kp0.shape[0], cap)
        info = plan.info()
        q = dev(np.ascontiguousarray(q_all[:, :n]))
        out = torch.empty((N, n, Hq, d), device="cuda")
        lse = torch.empty((N, n, Hq), device="cuda")
        kv = pref_bytes + N * n * 2 * Hkv * d * 2
        flop = 4.0 * Hq * N * n * Lp * d
        t, ts = timed(lambda i: plan.prefill(q, reps[i % R][0], reps[i % R][1], skd, svd, len0, out, lse))
        tp, tsp = timed(lambda i: pplan.prefill_paged(q, preps[i % R][0], preps[i % R][1], tab, len0, out, lse))
        res[f"n{n}"] = {"us_per_call": t * 1e6, "us_per_token": t * 1e6 / (N * n), "effective_kv_gbps": kv / t / 1e9,
                        "hbm_peak_frac": kv / t / 8e12, "tflops": flop / t / 1e12, "mfma_bf16_peak_frac": flop / t / 2.5e15,
                        "units": info.n_units, "blocks": info.n_blocks, "trials_us": [x * 1e6 for x in ts],
                        "paged": {"us_per_call": tp * 1e6, "us_per_token": tp * 1e6 / (N * n),
                                  "effective_kv_gbps": kv / tp / 1e9, "tflops": flop / tp / 1e12,
                                  "trials_us": [x * 1e6 for x in tsp]}}
        log(f"[bench] prefill n={n}: {t * 1e6:.1f} us per call ({t * 1e6 / (N * n):.2f} us/token), "
            f"{kv / t / 1e9:.0f} GB/s ({kv / t / 8e12:.1%} of 8 TB/s), {flop / t / 1e12:.0f} TFLOP/s "
            f"({flop / t / 2.5e15:.1%} of 2.5 PFLOP/s); {info.n_units} units, {info.n_blocks} blocks; "
            f"paged {tp * 1e6:.1f} us per call")
        del plan, pplan
    del reps, preps
    return res


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: fork-aware decode attention is not sharded across GPUs here "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch
    import oracle
    from paper_2608_13667_amd import forkattn as fa
    from paper_2608_13667_amd import workloads as W

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)

    if args.yardstick_copy:
        src = torch.ones(64 << 20, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    ns = tuple(int(x) for x in args.prefill_tokens.split(",") if x)
    if args.prefill_only:
        print(json.dumps({"instruction_prefill": prefill_timing(torch, fa, W, ns, args.trials)}), flush=True)
        return

    main_b = Bench(torch, fa, W, args.workload, args)
    K = args.steps if args.steps is not None else main_b.default_steps()
    if main_b.appends and math.ceil(K / main_b.R) > main_b.spec.steps:
        sys.exit(f"--steps {K} over {main_b.R} replicas exceeds the {main_b.spec.steps} appends each suffix buffer holds")
    rec = main_b.measure(K, args.warmup, args.trials, naive=not args.no_naive, mall_warm=True)
    main_bytes = main_b.kvb["total"]
    cpu = None
    if not args.no_cpu:
        cpu = cpu_oracle(oracle, main_b.w, main_b.n_seq, main_b.spec.n_q_heads, args.cpu_seconds)
    lifecycle = None
    if args.lifecycle and not main_b.paged:
        lifecycle = lifecycle_timing(fa, torch, main_b.w)
    main_b.release()

    subs = {}
    for name in [s for s in args.sub.split(",") if s and s != args.workload]:
        b = Bench(torch, fa, W, name, args)
        k = args.steps if args.steps is not None else b.default_steps()
        if b.appends:
            k = min(k, 256 * b.R)
        subs[name] = b.measure(k, args.warmup, args.trials, naive=not args.no_naive)
        b.release()
        del b

    prefill = None
    if not args.no_prefill:
        prefill = prefill_timing(torch, fa, W, ns, args.trials)

    probe = None
    if not args.no_probe:
        probe = read_probe(torch, fa, {"main_workload_bytes": main_bytes, "1GiB": 1 << 30})

    res = {
        "metric": "fork-decode attention steps/s and effective KV GB/s (% of HBM peak), 1 GPU",
        "value": rec["steps_per_s"],
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": rec["us_per_step"] / 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": rec["config"],
        "trials": args.trials,
        "trials_us_per_step": rec["trials_us_per_step"],
        "effective_kv_gbps": rec["effective_kv_gbps"],
        "hbm_peak_frac": rec["hbm_peak_frac"],
        "roofline": rec["roofline"],
        "cpu_baseline": cpu,
    }
    for key in ("naive_per_branch", "mall_warm_single_replica"):
        if key in rec:
            res[key] = rec[key]
    if probe:
        res["read_probe"] = probe
        best = max(p["gbps"] for p in probe.values())
        res["achievable_read_frac"] = {"step": rec["effective_kv_gbps"] / best,
                                       "partial_kernel": rec["roofline"]["achieved"] / best}
    res["sub_workloads"] = subs
    if prefill:
        res["instruction_prefill"] = prefill
    if lifecycle:
        res["lifecycle"] = lifecycle
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
