"""Helpers for GPU tests: move seeded workloads to the device and run the library on them."""
import numpy as np
import torch


def dev_bf16(bits: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def dev_i32(a: np.ndarray) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a, np.int32)).cuda()


def contig_plan(fa, w, share_prefix=True, rounds=0, max_suffix_len=None, blocks=0):
    s = w.spec
    msl = w.suffix_cap if max_suffix_len is None else max_suffix_len
    return fa.Plan.contig(s.n_q_heads, s.n_kv_heads, s.head_dim, w.n_branches, w.prefix_len, w.suffix_cap, msl,
                          share_prefix=share_prefix, rounds=rounds, blocks=blocks)


def to_dev_contig(w) -> dict:
    return dict(q=dev_bf16(w.q), prefix_k=dev_bf16(w.prefix_k), prefix_v=dev_bf16(w.prefix_v),
                suffix_k=dev_bf16(w.suffix_k), suffix_v=dev_bf16(w.suffix_v), suffix_len=dev_i32(w.suffix_len))


def run_contig(plan, dv, rows_hq):
    N, Hq, d = dv["q"].shape
    out = torch.full((N, Hq, d), float("nan"), device="cuda")
    lse = torch.full((N, Hq), float("nan"), device="cuda")
    plan.decode(dv["q"], dv["prefix_k"], dv["prefix_v"], dv["suffix_k"], dv["suffix_v"], dv["suffix_len"], out, lse)
    torch.cuda.synchronize()
    return out.cpu().numpy(), lse.cpu().numpy()


def paged_plan(fa, w, share_prefix=True, rounds=0, max_suffix_len=None, blocks=0):
    s = w.spec
    msl = int(w.suffix_len.max()) + s.page_headroom if max_suffix_len is None else max_suffix_len
    return fa.Plan.paged_plan(s.n_q_heads, s.n_kv_heads, s.head_dim, w.group_start, w.prefix_len,
                              w.page_table.shape[1], w.k_pool.shape[0], msl, share_prefix=share_prefix,
                              rounds=rounds, blocks=blocks)


def to_dev_paged(w) -> dict:
    return dict(q=dev_bf16(w.q), k_pool=dev_bf16(w.k_pool), v_pool=dev_bf16(w.v_pool),
                page_table=dev_i32(w.page_table), suffix_len=dev_i32(w.suffix_len))


def run_paged(plan, dv):
    S, Hq, d = dv["q"].shape
    out = torch.full((S, Hq, d), float("nan"), device="cuda")
    lse = torch.full((S, Hq), float("nan"), device="cuda")
    plan.decode_paged(dv["q"], dv["k_pool"], dv["v_pool"], dv["page_table"], dv["suffix_len"], out, lse)
    torch.cuda.synchronize()
    return out.cpu().numpy(), lse.cpu().numpy()
