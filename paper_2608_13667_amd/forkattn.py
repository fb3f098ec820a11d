"""ctypes binding of libforkattn.so (include/forkattn.h), argument marshalling only.

Every step of the computation runs in the library's HIP kernels; this module
turns torch device tensors into raw pointers and the current torch stream into a
hipStream_t.  Importing it fails loudly when the library has not been built.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Optional

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libforkattn.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is not built: run paper_2608_13667_amd.build.build() "
                      "(or __graft_entry__.build()) first")
_lib = C.CDLL(LIB_PATH)

FKA_OK, FKA_ERR_INVALID_ARG, FKA_ERR_UNSUPPORTED, FKA_ERR_HIP, FKA_ERR_NOMEM = 0, -1, -2, -3, -4
ERR_SUFFIX_CLAMPED, ERR_APPEND_NO_ROOM, ERR_BAD_PAGE, ERR_BAD_SCHEDULE = 1, 2, 4, 8


class Heads(C.Structure):
    _fields_ = [("n_q_heads", C.c_int32), ("n_kv_heads", C.c_int32), ("head_dim", C.c_int32),
                ("softmax_scale", C.c_float)]


class ContigDesc(C.Structure):
    _fields_ = [("n_branches", C.c_int32), ("prefix_len", C.c_int32), ("suffix_cap", C.c_int32),
                ("max_suffix_len", C.c_int32), ("share_prefix", C.c_int32), ("rounds", C.c_int32),
                ("blocks", C.c_int32)]


class PagedDesc(C.Structure):
    _fields_ = [("n_seqs", C.c_int32), ("n_groups", C.c_int32), ("page_size", C.c_int32),
                ("max_pages_per_seq", C.c_int32), ("n_pool_pages", C.c_int32), ("max_suffix_len", C.c_int32),
                ("share_prefix", C.c_int32), ("rounds", C.c_int32), ("blocks", C.c_int32)]


class PrefillDesc(C.Structure):
    _fields_ = [("n_branches", C.c_int32), ("n_tokens", C.c_int32), ("prefix_len", C.c_int32),
                ("suffix_cap", C.c_int32), ("max_suffix_len", C.c_int32), ("blocks", C.c_int32)]


class PrefillPagedDesc(C.Structure):
    _fields_ = [("n_branches", C.c_int32), ("n_tokens", C.c_int32), ("prefix_len", C.c_int32),
                ("page_size", C.c_int32), ("max_pages_per_seq", C.c_int32), ("n_pool_pages", C.c_int32),
                ("max_suffix_len", C.c_int32), ("blocks", C.c_int32)]


class PlanInfo(C.Structure):
    _fields_ = [("n_items", C.c_int32), ("n_units", C.c_int32), ("waves_per_block", C.c_int32),
                ("n_blocks", C.c_int32), ("rounds", C.c_int32), ("n_slots", C.c_int32), ("slot_rows", C.c_int32),
                ("static_split", C.c_int32), ("units_per_block", C.c_int32),
                ("workspace_bytes", C.c_size_t)]


class Slot(C.Structure):
    _fields_ = [("slot", C.c_int32), ("seq0", C.c_int32), ("nseq", C.c_int32), ("kv_head", C.c_int32),
                ("rows", C.c_int32), ("prefix_begin", C.c_int32), ("prefix_end", C.c_int32),
                ("suffix_begin", C.c_int32), ("suffix_end", C.c_int32), ("prefix_len", C.c_int32)]


_vp = C.c_void_p
_sig = {
    "fka_version": ([], C.c_int),
    "fka_last_error": ([], C.c_char_p),
    "fka_plan_create_contig": ([C.POINTER(Heads), C.POINTER(ContigDesc), C.POINTER(_vp)], C.c_int),
    "fka_plan_create_paged": ([C.POINTER(Heads), C.POINTER(PagedDesc), _vp, _vp, C.POINTER(_vp)], C.c_int),
    "fka_fork_decode": ([_vp] * 10, C.c_int),
    "fka_append_kv": ([_vp] * 7, C.c_int),
    "fka_fork_step": ([_vp] * 12, C.c_int),
    "fka_fork_decode_paged": ([_vp] * 9, C.c_int),
    "fka_fork_step_paged": ([_vp] * 11, C.c_int),
    "fka_append_kv_paged": ([_vp] * 8, C.c_int),
    "fka_gather_paged": ([_vp, C.c_int32, _vp, _vp, _vp, C.c_int32, _vp, _vp, _vp], C.c_int),
    "fka_gather_paged_range": ([_vp, C.c_int32, C.c_int32, C.c_int32, _vp, _vp, _vp, _vp, _vp, _vp], C.c_int),
    "fka_plan_get_info": ([_vp, C.POINTER(PlanInfo)], C.c_int),
    "fka_plan_create_prefill": ([C.POINTER(Heads), C.POINTER(PrefillDesc), C.POINTER(_vp)], C.c_int),
    "fka_prefill": ([_vp] * 10, C.c_int),
    "fka_plan_create_prefill_paged": ([C.POINTER(Heads), C.POINTER(PrefillPagedDesc), C.POINTER(_vp)], C.c_int),
    "fka_prefill_paged": ([_vp] * 9, C.c_int),
    "fka_fork_decode_noalloc": ([C.POINTER(Heads), C.POINTER(ContigDesc)] + [_vp] * 10, C.c_int),
    "fka_plan_slots": ([_vp, _vp, _vp, C.c_int32, C.POINTER(C.c_int32)], C.c_int),
    "fka_partials": ([_vp] * 10, C.c_int),
    "fka_partials_paged": ([_vp] * 9, C.c_int),
    "fka_lse_merge": ([C.c_int32, C.c_int32, C.c_int32, _vp, _vp, _vp, _vp, _vp], C.c_int),
    "fka_plan_device_error": ([_vp, C.POINTER(C.c_int32)], C.c_int),
    "fka_read_probe": ([_vp, C.c_size_t, C.c_int32, C.c_int32, C.c_int32, _vp, _vp], C.c_int),
    "fka_plan_destroy": ([_vp], None),
    "fka_pool_create": ([C.c_int32, C.POINTER(_vp)], C.c_int),
    "fka_pool_destroy": ([_vp], None),
    "fka_pool_free_pages": ([_vp], C.c_int32),
    "fka_pool_refcount": ([_vp, C.c_int32], C.c_int32),
    "fka_pool_alloc": ([_vp, C.c_int32, _vp], C.c_int),
    "fka_pool_retain": ([_vp, C.c_int32, _vp], C.c_int),
    "fka_pool_release": ([_vp, C.c_int32, _vp], C.c_int),
    "fka_pool_fork": ([_vp, _vp, C.c_int32, _vp, C.c_int32, C.c_int32, C.c_int32], C.c_int),
    "fka_pool_reserve": ([_vp, _vp, C.c_int32, C.c_int32, C.c_int32, C.c_int32, C.POINTER(C.c_int32)], C.c_int),
    "fka_pool_drop": ([_vp, _vp, C.c_int32, C.c_int32], C.c_int),
    "fka_pool_promote": ([_vp, _vp, C.c_int32, C.c_int32, C.c_int32, C.c_int32, _vp, C.POINTER(C.c_int32)],
                         C.c_int),
    "fka_scatter_pages": ([_vp, _vp, C.c_int32, C.c_int32, _vp, C.c_int32, C.c_int32, C.c_int32, _vp, _vp, _vp, _vp],
                          C.c_int),
}
for _name, (_args, _res) in _sig.items():
    _f = getattr(_lib, _name)
    _f.argtypes = _args
    _f.restype = _res

EXPORTED = tuple(_sig)


class FkaError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"status {status}: {msg}")
        self.status = status


def _check(status: int):
    if status != FKA_OK:
        raise FkaError(status, _lib.fka_last_error().decode())


def last_error() -> str:
    return _lib.fka_last_error().decode()


def version() -> int:
    return _lib.fka_version()


_KIND_DTYPES = {"bf16": torch.bfloat16, "i32": torch.int32, "f32": torch.float32}


def _p(t: Optional[torch.Tensor], kind: Optional[str] = None, device: Optional[int] = None):
    """Device pointer of a contiguous tensor on the plan's GPU, of the dtype the C ABI expects
    for this argument (bf16 q/K/V, int32 lengths and page tables, fp32 outputs)."""
    if t is None:
        return None
    if not isinstance(t, torch.Tensor):
        raise ValueError("expected a torch tensor")
    if not t.is_cuda:
        raise ValueError("tensor must be on the GPU (the library reads device memory)")
    if device is not None and t.get_device() != device:
        raise ValueError(f"tensor is on cuda:{t.get_device()}, the plan's device is cuda:{device}")
    if kind is not None and t.dtype != _KIND_DTYPES[kind]:
        raise ValueError(f"tensor must be {kind}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError("tensor must be contiguous")
    return _vp(t.data_ptr())


def _stream(stream) -> _vp:
    if stream is None:
        stream = torch.cuda.current_stream()
    return _vp(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


class Plan:
    """A fork plan: the static work schedule and the device workspace (see fka_plan_create_*)."""

    def __init__(self, handle: int, paged: bool, heads: Heads, n_seqs: int):
        self._h = _vp(handle)
        self.device = torch.cuda.current_device() if torch.cuda.is_available() else None
        self.paged = paged
        self.heads = heads
        self.n_seqs = n_seqs

    @classmethod
    def contig(cls, n_q_heads, n_kv_heads, head_dim, n_branches, prefix_len, suffix_cap, max_suffix_len,
               share_prefix=True, rounds=0, softmax_scale=0.0, blocks=0) -> "Plan":
        h = Heads(n_q_heads, n_kv_heads, head_dim, softmax_scale)
        d = ContigDesc(n_branches, prefix_len, suffix_cap, max_suffix_len, int(bool(share_prefix)), rounds, blocks)
        out = _vp()
        _check(_lib.fka_plan_create_contig(C.byref(h), C.byref(d), C.byref(out)))
        return cls(out.value, False, h, n_branches)

    @classmethod
    def paged_plan(cls, n_q_heads, n_kv_heads, head_dim, group_start, group_prefix_len, max_pages_per_seq,
                   n_pool_pages, max_suffix_len, share_prefix=True, rounds=0, softmax_scale=0.0,
                   page_size=16, blocks=0) -> "Plan":
        gs = np.ascontiguousarray(group_start, np.int32)
        gl = np.ascontiguousarray(group_prefix_len, np.int32)
        h = Heads(n_q_heads, n_kv_heads, head_dim, softmax_scale)
        d = PagedDesc(int(gs[-1]), len(gl), page_size, max_pages_per_seq, n_pool_pages, max_suffix_len,
                      int(bool(share_prefix)), rounds, blocks)
        out = _vp()
        _check(_lib.fka_plan_create_paged(C.byref(h), C.byref(d), gs.ctypes.data_as(_vp), gl.ctypes.data_as(_vp),
                                          C.byref(out)))
        return cls(out.value, True, h, int(gs[-1]))

    @classmethod
    def prefill_plan(cls, n_q_heads, n_kv_heads, head_dim, n_branches, n_tokens, prefix_len, suffix_cap,
                     max_suffix_len, softmax_scale=0.0, blocks=0) -> "Plan":
        """An instruction-prefill plan (fka_plan_create_prefill): n_tokens per branch."""
        h = Heads(n_q_heads, n_kv_heads, head_dim, softmax_scale)
        d = PrefillDesc(n_branches, n_tokens, prefix_len, suffix_cap, max_suffix_len, blocks)
        out = _vp()
        _check(_lib.fka_plan_create_prefill(C.byref(h), C.byref(d), C.byref(out)))
        return cls(out.value, False, h, n_branches * n_tokens)

    @classmethod
    def prefill_paged_plan(cls, n_q_heads, n_kv_heads, head_dim, n_branches, n_tokens, prefix_len, max_pages_per_seq,
                           n_pool_pages, max_suffix_len, softmax_scale=0.0, blocks=0, page_size=16) -> "Plan":
        """A paged instruction-prefill plan (fka_plan_create_prefill_paged): n_tokens per branch."""
        h = Heads(n_q_heads, n_kv_heads, head_dim, softmax_scale)
        d = PrefillPagedDesc(n_branches, n_tokens, prefix_len, page_size, max_pages_per_seq, n_pool_pages,
                             max_suffix_len, blocks)
        out = _vp()
        _check(_lib.fka_plan_create_prefill_paged(C.byref(h), C.byref(d), C.byref(out)))
        return cls(out.value, True, h, n_branches * n_tokens)

    def prefill_paged(self, q, k_pool, v_pool, page_table, suffix_len, out, out_lse=None, stream=None):
        """fka_prefill_paged: q bf16 [N][n][Hq][d], page_table int32 [N][max_pages] -> out fp32 [N][n][Hq][d]."""
        d = self.device
        _check(_lib.fka_prefill_paged(self._h, _p(q, "bf16", d), _p(k_pool, "bf16", d), _p(v_pool, "bf16", d),
                                      _p(page_table, "i32", d), _p(suffix_len, "i32", d), _p(out, "f32", d),
                                      _p(out_lse, "f32", d), _stream(stream)))

    def prefill(self, q, prefix_k, prefix_v, suffix_k, suffix_v, suffix_len, out, out_lse=None, stream=None):
        """fka_prefill: q bf16 [N][n][Hq][d] -> out fp32 [N][n][Hq][d], out_lse fp32 [N][n][Hq]."""
        d = self.device
        _check(_lib.fka_prefill(self._h, _p(q, "bf16", d), _p(prefix_k, "bf16", d), _p(prefix_v, "bf16", d),
                                _p(suffix_k, "bf16", d), _p(suffix_v, "bf16", d), _p(suffix_len, "i32", d),
                                _p(out, "f32", d), _p(out_lse, "f32", d), _stream(stream)))

    def close(self):
        if self._h is not None and self._h.value:
            _lib.fka_plan_destroy(self._h)
        self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    @property
    def handle(self):
        return self._h

    def info(self) -> PlanInfo:
        i = PlanInfo()
        _check(_lib.fka_plan_get_info(self._h, C.byref(i)))
        return i

    def slots(self, suffix_len) -> list:
        """The partial slots a decode writes for these (host) suffix lengths (fka_plan_slots)."""
        import numpy as np
        sl = np.ascontiguousarray(suffix_len, np.int32)
        if sl.shape != (self.n_seqs,):
            raise ValueError(f"suffix_len must have shape ({self.n_seqs},)")
        n = C.c_int32(0)
        _check(_lib.fka_plan_slots(self._h, sl.ctypes.data_as(_vp), None, 0, C.byref(n)))
        arr = (Slot * max(1, n.value))()
        _check(_lib.fka_plan_slots(self._h, sl.ctypes.data_as(_vp), C.cast(arr, _vp), n.value, C.byref(n)))
        return [{f: getattr(arr[i], f) for f, _ in Slot._fields_} for i in range(n.value)]

    def device_error(self) -> int:
        v = C.c_int32(0)
        _check(_lib.fka_plan_device_error(self._h, C.byref(v)))
        return v.value

    # ---- contiguous
    def decode(self, q, prefix_k, prefix_v, suffix_k, suffix_v, suffix_len, out, out_lse=None, stream=None):
        d = self.device
        _check(_lib.fka_fork_decode(self._h, _p(q, "bf16", d), _p(prefix_k, "bf16", d), _p(prefix_v, "bf16", d),
                                    _p(suffix_k, "bf16", d), _p(suffix_v, "bf16", d), _p(suffix_len, "i32", d),
                                    _p(out, "f32", d), _p(out_lse, "f32", d), _stream(stream)))

    def append(self, k_new, v_new, suffix_k, suffix_v, suffix_len, stream=None):
        d = self.device
        _check(_lib.fka_append_kv(self._h, _p(k_new, "bf16", d), _p(v_new, "bf16", d), _p(suffix_k, "bf16", d),
                                  _p(suffix_v, "bf16", d), _p(suffix_len, "i32", d), _stream(stream)))

    def step(self, q, k_new, v_new, prefix_k, prefix_v, suffix_k, suffix_v, suffix_len, out, out_lse=None,
             stream=None):
        d = self.device
        _check(_lib.fka_fork_step(self._h, _p(q, "bf16", d), _p(k_new, "bf16", d), _p(v_new, "bf16", d),
                                  _p(prefix_k, "bf16", d), _p(prefix_v, "bf16", d), _p(suffix_k, "bf16", d),
                                  _p(suffix_v, "bf16", d), _p(suffix_len, "i32", d), _p(out, "f32", d),
                                  _p(out_lse, "f32", d), _stream(stream)))

    def partials(self, q, prefix_k, prefix_v, suffix_k, suffix_v, suffix_len, part_o, part_lse, stream=None):
        d = self.device
        _check(_lib.fka_partials(self._h, _p(q, "bf16", d), _p(prefix_k, "bf16", d), _p(prefix_v, "bf16", d),
                                 _p(suffix_k, "bf16", d), _p(suffix_v, "bf16", d), _p(suffix_len, "i32", d),
                                 _p(part_o, "f32", d), _p(part_lse, "f32", d), _stream(stream)))

    # ---- paged
    def partials_paged(self, q, k_pool, v_pool, page_table, suffix_len, part_o, part_lse, stream=None):
        d = self.device
        _check(_lib.fka_partials_paged(self._h, _p(q, "bf16", d), _p(k_pool, "bf16", d), _p(v_pool, "bf16", d),
                                       _p(page_table, "i32", d), _p(suffix_len, "i32", d), _p(part_o, "f32", d),
                                       _p(part_lse, "f32", d), _stream(stream)))

    def decode_paged(self, q, k_pool, v_pool, page_table, suffix_len, out, out_lse=None, stream=None):
        d = self.device
        _check(_lib.fka_fork_decode_paged(self._h, _p(q, "bf16", d), _p(k_pool, "bf16", d), _p(v_pool, "bf16", d),
                                          _p(page_table, "i32", d), _p(suffix_len, "i32", d), _p(out, "f32", d),
                                          _p(out_lse, "f32", d), _stream(stream)))

    def step_paged(self, q, k_new, v_new, k_pool, v_pool, page_table, suffix_len, out, out_lse=None, stream=None):
        d = self.device
        _check(_lib.fka_fork_step_paged(self._h, _p(q, "bf16", d), _p(k_new, "bf16", d), _p(v_new, "bf16", d),
                                        _p(k_pool, "bf16", d), _p(v_pool, "bf16", d), _p(page_table, "i32", d),
                                        _p(suffix_len, "i32", d), _p(out, "f32", d), _p(out_lse, "f32", d),
                                        _stream(stream)))

    def append_paged(self, k_new, v_new, k_pool, v_pool, page_table, suffix_len, stream=None):
        d = self.device
        _check(_lib.fka_append_kv_paged(self._h, _p(k_new, "bf16", d), _p(v_new, "bf16", d), _p(k_pool, "bf16", d),
                                        _p(v_pool, "bf16", d), _p(page_table, "i32", d), _p(suffix_len, "i32", d),
                                        _stream(stream)))

    def gather_paged_range(self, seq, begin, out_len, k_pool, v_pool, page_table, k_out, v_out, stream=None):
        d = self.device
        _check(_lib.fka_gather_paged_range(self._h, int(seq), int(begin), int(out_len), _p(k_pool, "bf16", d),
                                           _p(v_pool, "bf16", d), _p(page_table, "i32", d), _p(k_out, "bf16", d),
                                           _p(v_out, "bf16", d), _stream(stream)))

    def gather_paged(self, seq, k_pool, v_pool, page_table, out_len, k_out, v_out, stream=None):
        d = self.device
        _check(_lib.fka_gather_paged(self._h, int(seq), _p(k_pool, "bf16", d), _p(v_pool, "bf16", d),
                                     _p(page_table, "i32", d), int(out_len), _p(k_out, "bf16", d),
                                     _p(v_out, "bf16", d), _stream(stream)))


def _host_i32(a: np.ndarray) -> _vp:
    if a.dtype != np.int32 or not a.flags["C_CONTIGUOUS"] or not a.flags["WRITEABLE"]:
        raise ValueError("host page ids must be a writeable C-contiguous int32 array")
    return _vp(a.ctypes.data)


class Pool:
    """Page pool of a paged K/V store (host bookkeeping; see fka_pool_* in forkattn.h).  Page
    tables are host numpy int32 arrays [rows][max_pages] with -1 for no page."""

    def __init__(self, n_pages: int):
        h = _vp()
        _check(_lib.fka_pool_create(int(n_pages), C.byref(h)))
        self._h = h

    def close(self):
        if self._h:
            _lib.fka_pool_destroy(self._h)
            self._h = _vp()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def free_pages(self) -> int:
        return _lib.fka_pool_free_pages(self._h)

    def refcount(self, page: int) -> int:
        return _lib.fka_pool_refcount(self._h, int(page))

    def alloc(self, n: int) -> np.ndarray:
        ids = np.empty(int(n), np.int32)
        _check(_lib.fka_pool_alloc(self._h, int(n), _host_i32(ids)))
        return ids

    def retain(self, ids: np.ndarray):
        ids = np.ascontiguousarray(ids, np.int32)
        _check(_lib.fka_pool_retain(self._h, ids.size, _host_i32(ids)))

    def release(self, ids: np.ndarray):
        ids = np.ascontiguousarray(ids, np.int32)
        _check(_lib.fka_pool_release(self._h, ids.size, _host_i32(ids)))

    def fork(self, prefix_pages: np.ndarray, table: np.ndarray, first: int, n: int):
        prefix_pages = np.ascontiguousarray(prefix_pages, np.int32)
        _check(_lib.fka_pool_fork(self._h, _host_i32(prefix_pages), prefix_pages.size, _host_i32(table),
                                  table.shape[1], int(first), int(n)))

    def reserve(self, table: np.ndarray, seq: int, prefix_len: int, suffix_len: int) -> int:
        n_new = C.c_int32(0)
        _check(_lib.fka_pool_reserve(self._h, _host_i32(table), table.shape[1], int(seq), int(prefix_len),
                                     int(suffix_len), C.byref(n_new)))
        return n_new.value

    def drop(self, table: np.ndarray, seq: int):
        _check(_lib.fka_pool_drop(self._h, _host_i32(table), table.shape[1], int(seq)))

    def promote(self, table: np.ndarray, seq: int, prefix_len: int, suffix_len: int):
        """Returns (dense page ids, first position to rewrite)."""
        n = (int(prefix_len) + int(suffix_len) + 15) // 16
        dense = np.full(max(n, 1), -1, np.int32)
        frm = C.c_int32(0)
        _check(_lib.fka_pool_promote(self._h, _host_i32(table), table.shape[1], int(seq), int(prefix_len),
                                     int(suffix_len), _host_i32(dense), C.byref(frm)))
        return dense[:n], frm.value


def scatter_pages(k_src, v_src, frm, page_row, n_pool_pages, k_pool, v_pool, err=None, stream=None):
    """Positions [frm, frm + n) held in k_src / v_src bf16 [Hkv][n][d] -> pool pages of page_row (device int32)."""
    Hkv, n, d = k_src.shape
    _check(_lib.fka_scatter_pages(_p(k_src, "bf16"), _p(v_src, "bf16"), int(frm) + n, int(frm), _p(page_row, "i32"), Hkv, d, int(n_pool_pages),
                                  _p(k_pool, "bf16"), _p(v_pool, "bf16"), _p(err, "i32"), _stream(stream)))


def read_probe(buf, blocks, threads, unroll, sink, stream=None):
    """Read-only streaming probe over the device tensor buf (fka_read_probe)."""
    _check(_lib.fka_read_probe(_p(buf), buf.numel() * buf.element_size(), int(blocks), int(threads), int(unroll),
                               _p(sink), _stream(stream)))


def decode_noalloc(n_q_heads, n_kv_heads, head_dim, prefix_len, suffix_cap, max_suffix_len, q, prefix_k, prefix_v,
                   suffix_k, suffix_v, suffix_len, out, out_lse=None, err=None, rounds=0, softmax_scale=0.0, blocks=0,
                   stream=None):
    """fka_fork_decode_noalloc: a shared-prefix decode without a plan, on the library's static scratch
    (the sizes are those of Plan.contig with share_prefix=True; n_branches is q's first dimension)."""
    dev = q.get_device() if isinstance(q, torch.Tensor) and q.is_cuda else None
    h = Heads(n_q_heads, n_kv_heads, head_dim, softmax_scale)
    d = ContigDesc(q.shape[0], prefix_len, suffix_cap, max_suffix_len, 1, rounds, blocks)
    _check(_lib.fka_fork_decode_noalloc(C.byref(h), C.byref(d), _p(q, "bf16", dev), _p(prefix_k, "bf16", dev),
                                        _p(prefix_v, "bf16", dev), _p(suffix_k, "bf16", dev), _p(suffix_v, "bf16", dev),
                                        _p(suffix_len, "i32", dev), _p(out, "f32", dev), _p(out_lse, "f32", dev),
                                        _p(err, "i32", dev), _stream(stream)))


def lse_merge(part_o, part_lse, out, out_lse=None, stream=None):
    """part_o fp32 [P][R][d], part_lse fp32 [P][R] -> out fp32 [R][d], out_lse fp32 [R]."""
    P, R, d = part_o.shape
    _check(_lib.fka_lse_merge(R, P, d, _p(part_o, "f32"), _p(part_lse, "f32"), _p(out, "f32"), _p(out_lse, "f32"), _stream(stream)))


def raw_call(name: str, *args) -> int:
    """Call an exported function with raw ctypes arguments; returns its status (for ABI tests)."""
    return getattr(_lib, name)(*args)
