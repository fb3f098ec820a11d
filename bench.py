"""Fork-aware decode attention benchmark (one GPU).

A step is one fork-decode step of one attention layer: every sequence of the fork
(main thread + 4 branches) appends its new K/V token and attends with one new query
over the shared prefix and its own suffix.  The default workload is the long agent
context: 32768-token shared prefix, 5 sequences, 40 query / 8 KV heads, head_dim 128,
suffixes of 512..2048 tokens, 256 appended tokens per layer.  Layers are replicated
so that the working set (>= 1 GiB) exceeds the 256 MB Infinity Cache and every step
reads HBM; step i runs on replica i % R.  Inputs are resident in HBM before the timed
region.  Prints one JSON line.
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
COPY_PROBE_BYTES = 256 << 20
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")
KERNEL_SOURCE = os.path.join(ROOT, "paper_2608_13667_amd", "csrc", "partials.hip")


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
    ap.add_argument("--steps", type=int, default=None, help="timed steps (default: 256 appends per replica)")
    # 200 untimed steps: on the 128k-prefix workload the first ~20 ms of back-to-back launches run
    # a transient (steps 5-10% slower, then settling); shorter workloads are unaffected
    ap.add_argument("--warmup", type=int, default=200)
    ap.add_argument("--workload", default="long", choices=sorted(DESCRIPTIONS))
    ap.add_argument("--replicas", type=int, default=0, help="layer replicas (0: enough for >= 1 GiB)")
    ap.add_argument("--rounds", type=int, default=0, help="schedule rounds of the resident waves (0: automatic)")
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-naive", action="store_true", help="skip the naive per-branch GPU baseline")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--lifecycle", action="store_true",
                    help="also time the fork lifecycle on the page pool (contiguous workloads' shapes)")
    return ap.parse_args()


def lifecycle_timing(fa, torch, w):
    """One turn transition of the fork lifecycle at the workload's shape, with a page pool: fork
    the snapshot to all sequences, reserve their suffix pages, drop the branches, promote the main
    sequence (host bookkeeping), and the promote's device work (a gather of the main context's tail,
    from the first page the dense layout rewrites, and its scatter into the dense pages).  Host calls are timed with perf_counter over many cycles,
    the device work with HIP events on the launch stream."""
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
    # branch-instruction prefill, one chunk: n tokens per branch as N * n virtual sequences in one
    # group (token t of branch b reads b's pages with suffix length L_b + t + 1), as many as the
    # 64 query rows per KV head allow; the prefix is read once per chunk
    G = spec.n_q_heads // Hkv
    n = max(1, 64 // (N * G))
    table = np.full((N, max_pages), -1, np.int32)
    snap2 = pool.alloc(a)
    pool.fork(snap2, table, 0, N)
    for b in range(N):
        pool.reserve(table, b, Lp, min(lens[b] + n, max(lens)))
    vt = torch.from_numpy(np.repeat(table, n, axis=0)).cuda()
    vlen_np = np.array([min(lens[b] + t + 1, max(lens)) for b in range(N) for t in range(n)], np.int32)
    vlen = torch.from_numpy(vlen_np).cuda()
    pplan = fa.Plan.paged_plan(spec.n_q_heads, Hkv, d, [0, N * n], [Lp], max_pages, n_pages, max(lens))
    q = torch.zeros((N * n, spec.n_q_heads, d), dtype=torch.bfloat16, device="cuda")
    o = torch.empty((N * n, spec.n_q_heads, d), device="cuda")
    for _ in range(20):
        pplan.decode_paged(q, pages, v_pages, vt, vlen, o, None, stream)
    e0.record(stream)
    for _ in range(reps * 5):
        pplan.decode_paged(q, pages, v_pages, vt, vlen, o, None, stream)
    e1.record(stream)
    torch.cuda.synchronize()
    pf_s = e0.elapsed_time(e1) / 1e3 / (reps * 5)
    pf_bytes = per_tok * (Lp + sum(int(x) for x in vlen_np))  # the prefix once, each token's suffix
    pplan.close()
    pool.close()
    ms = lambda v: float(np.median(v) * 1e6)
    return {"tokens_promoted": L0, "host_us": {k: ms(v) for k, v in host.items()},
            "promote_device_us": dev_s * 1e6, "promote_device_gbps": moved / dev_s / 1e9,
            "prefill_chunk": {"tokens_per_branch": n, "us": pf_s * 1e6, "kv_gbps": pf_bytes / pf_s / 1e9}}


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
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()

    t0 = time.time()
    w = W.make(args.workload)
    spec = w.spec
    log(f"[bench] generated {args.workload} in {time.time() - t0:.1f}s")
    paged = spec.paged
    appends = spec.steps > 0
    if paged:
        kvb = W.kv_bytes_paged(w)
    else:
        kvb = W.kv_bytes_contig(w)
    R = args.replicas or max(1, math.ceil((1 << 30) / kvb["total"]))
    K = args.steps if args.steps is not None else (256 * R if appends else max(200, 20 * R))
    if appends and math.ceil(K / R) > spec.steps:
        sys.exit(f"--steps {K} over {R} replicas exceeds the {spec.steps} appends each suffix buffer holds")

    # device replicas of the layer (same values, distinct memory)
    per_tok = 2 * spec.n_kv_heads * spec.head_dim * 2
    if paged:
        base = dict(q=dev(w.q), k_pool=dev(w.k_pool), v_pool=dev(w.v_pool),
                    page_table=torch.from_numpy(w.page_table).cuda(), suffix_len=torch.from_numpy(w.suffix_len).cuda())
        reps = [base] + [{k: v.clone() for k, v in base.items()} for _ in range(R - 1)]

        def mk_plan(share):
            return fa.Plan.paged_plan(spec.n_q_heads, spec.n_kv_heads, spec.head_dim, w.group_start, w.prefix_len,
                                      w.page_table.shape[1], w.k_pool.shape[0], int(w.suffix_len.max()),
                                      share_prefix=share, rounds=args.rounds)
    else:
        base = dict(q=dev(w.q), prefix_k=dev(w.prefix_k), prefix_v=dev(w.prefix_v), suffix_k=dev(w.suffix_k),
                    suffix_v=dev(w.suffix_v), suffix_len=torch.from_numpy(w.suffix_len).cuda())
        reps = [base] + [{k: v.clone() for k, v in base.items()} for _ in range(R - 1)]

        def mk_plan(share):
            return fa.Plan.contig(spec.n_q_heads, spec.n_kv_heads, spec.head_dim, w.n_branches, w.prefix_len,
                                  w.suffix_cap, w.suffix_cap, share_prefix=share, rounds=args.rounds)
    n_seq = w.q.shape[0]
    out = torch.empty((n_seq, spec.n_q_heads, spec.head_dim), device="cuda")
    lse = torch.empty((n_seq, spec.n_q_heads), device="cuda")
    if appends:
        step_q, step_k, step_v = dev(w.step_q), dev(w.step_k), dev(w.step_v)
    len0 = torch.from_numpy(w.suffix_len).cuda()
    log(f"[bench] {R} replicas x {kvb['total'] / 2**20:.1f} MiB, {K} timed steps")

    def run(plan, i):
        r = reps[i % R]
        if paged:
            plan.decode_paged(r["q"], r["k_pool"], r["v_pool"], r["page_table"], r["suffix_len"], out, lse)
        elif appends:
            j = i // R
            plan.step(step_q[j], step_k[j], step_v[j], r["prefix_k"], r["prefix_v"], r["suffix_k"], r["suffix_v"],
                      r["suffix_len"], out, lse)
        else:
            plan.decode(r["q"], r["prefix_k"], r["prefix_v"], r["suffix_k"], r["suffix_v"], r["suffix_len"], out, lse)

    def reset():
        for r in reps:
            r["suffix_len"].copy_(len0)

    def timed_loop(plan, n_steps, warmup):
        reset()
        for i in range(warmup):
            run(plan, i)
        torch.cuda.synchronize()
        reset()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for i in range(n_steps):
            run(plan, i)
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) * 1e-3

    def step_bytes(n_steps):
        """Algorithmic K/V bytes of the timed loop: prefix once per step plus every suffix at its length."""
        total = 0
        sl0 = int(np.sum(w.suffix_len))
        for i in range(n_steps):
            extra = (i // R + 1) * n_seq if appends else 0
            total += kvb["prefix"] + (sl0 + extra) * per_tok
        return total

    plan = mk_plan(True)
    info = plan.info()
    secs = timed_loop(plan, K, args.warmup)
    assert plan.device_error() == 0
    alg = step_bytes(K)
    gbps = alg / secs / 1e9
    log(f"[bench] fork-aware: {K / secs:.1f} steps/s, {secs / K * 1e6:.2f} us/step, {gbps:.0f} GB/s")

    # dominant kernel alone: the partial-attention kernel, timed on the stream it runs on
    po = torch.empty((info.n_slots, info.slot_rows, spec.head_dim), device="cuda")
    pl = torch.empty((info.n_slots, info.slot_rows), device="cuda")
    reset()
    kp = max(50, min(K, 400))
    if not paged:
        def part(i):
            r = reps[i % R]
            plan.partials(r["q"], r["prefix_k"], r["prefix_v"], r["suffix_k"], r["suffix_v"], r["suffix_len"], po, pl)
        # as inside a step, the partial kernel runs on the schedule the previous launch cached: one
        # decode at these lengths (all replicas hold the same ones) builds it
        r0 = reps[0]
        plan.decode(r0["q"], r0["prefix_k"], r0["prefix_v"], r0["suffix_k"], r0["suffix_v"], r0["suffix_len"], out, lse)
        for i in range(5):
            part(i)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for i in range(kp):
            part(i)
        e1.record()
        torch.cuda.synchronize()
        k_secs = e0.elapsed_time(e1) * 1e-3 / kp
        k_bytes = kvb["total"]
        roof_name = "partials_kernel (prefix + suffix partial attention)"
    else:
        k_secs = secs / K
        k_bytes = kvb["total"]
        roof_name = "whole paged step (partials + merge)"
    k_gbps = k_bytes / k_secs / 1e9

    result_extra = {}
    if not args.no_naive:
        nplan = mk_plan(False)
        kn = max(R, K // 4)
        nsecs = timed_loop(nplan, kn, min(args.warmup, kn))
        nalg = step_bytes(kn)
        result_extra["naive_per_branch"] = {
            "steps_per_s": kn / nsecs, "us_per_step": nsecs / kn * 1e6,
            "effective_kv_gbps": nalg / nsecs / 1e9,
            "requested_kv_gbps": (nalg + (kvb["naive"] - kvb["total"]) * kn) / nsecs / 1e9,
            "prefix_reuse_speedup": (nsecs / kn) / (secs / K)}
        log(f"[bench] naive: {kn / nsecs:.1f} steps/s, speed-up of sharing {(nsecs / kn) / (secs / K):.2f}x")
        nplan.close()

    # MALL-warm single-replica figure (labelled: the working set fits in the 256 MB Infinity Cache)
    if not paged and kvb["total"] < MALL_BYTES:
        r0 = reps[0]
        reset()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        nw = min(K, 200)
        e0.record()
        for i in range(nw):
            plan.decode(r0["q"], r0["prefix_k"], r0["prefix_v"], r0["suffix_k"], r0["suffix_v"], r0["suffix_len"], out,
                        lse)
        e1.record()
        torch.cuda.synchronize()
        ws = e0.elapsed_time(e1) * 1e-3
        result_extra["mall_warm_single_replica"] = {"steps_per_s": nw / ws, "kv_gbps": kvb["total"] * nw / ws / 1e9}

    # context probes: a plain 256 MiB device copy (its FETCH_SIZE / WRITE_SIZE counters are the
    # yardstick that turns counter readings into bytes) and its achieved copy bandwidth
    x = torch.empty(COPY_PROBE_BYTES // 4, dtype=torch.float32, device="cuda").fill_(1.0)
    y = torch.empty_like(x)
    y.copy_(x)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(10):
        y.copy_(x)
    e1.record()
    torch.cuda.synchronize()
    result_extra["copy_probe_gbps"] = 10 * 2 * COPY_PROBE_BYTES / (e0.elapsed_time(e1) * 1e-3) / 1e9
    del x, y

    cpu = None
    if not args.no_cpu:
        oracle.build(force=False)
        t_start = time.time()
        n = 0
        while True:
            oracle.decode_workload(w)
            n += 1
            if time.time() - t_start >= args.cpu_seconds:
                break
        cs = time.time() - t_start
        cpu = {"value": n / cs, "unit": "steps/s", "cores": oracle.threads(), "kind": "oracle",
               "sample": f"{n} full decode steps (all {n_seq} x {spec.n_q_heads} rows) at the initial lengths, "
                         f"fp64 on the host"}
        log(f"[bench] cpu oracle: {n / cs:.3f} steps/s on {cpu['cores']} threads")

    cfg = {"workload": DESCRIPTIONS[args.workload], "name": args.workload, "replicas": R,
           "working_set_gib": R * kvb["total"] / 2**30, "blocks": info.n_blocks,
           "waves_per_block": info.waves_per_block, "rounds": info.rounds, "work_items": info.n_items}
    res = {
        "metric": "fork-decode attention steps/s and effective KV GB/s (% of HBM peak), 1 GPU",
        "value": K / secs,
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": secs / K * 1e3,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": cfg,
        "effective_kv_gbps": gbps,
        "hbm_peak_frac": gbps / HBM_PEAK_GBPS,
        "roofline": {"bound": "hbm", "kernel": roof_name, "achieved": k_gbps, "peak": HBM_PEAK_GBPS, "unit": "GB/s",
                     "frac": k_gbps / HBM_PEAK_GBPS, "traffic": measured_traffic(args.workload),
                     "avg_launch_us": k_secs * 1e6, "bytes_per_launch": k_bytes},
        "cpu_baseline": cpu,
    }
    res.update(result_extra)
    if args.lifecycle and not paged:
        res["lifecycle"] = lifecycle_timing(fa, torch, w)
        log(f"[bench] lifecycle: {res['lifecycle']}")
    plan.close()
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
