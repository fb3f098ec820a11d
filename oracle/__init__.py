"""Python face of the fp64 CPU oracle (test infrastructure only).

Only the tests, the smoke check and the benchmark's CPU-baseline leg use this
package; the product path never does.  ``build()`` compiles ``oracle.c`` with gcc
into ``liboracle.so`` next to it; the wrappers below marshal numpy arrays (bf16
bit patterns as uint16) into it and return fp64 results.  The C file states what
is computed and which passage of the paper each function follows.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile the oracle with gcc (OpenMP, strict IEEE fp64: no fast-math)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11", _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            build()
        lib = C.CDLL(_LIB)
        p = C.c_void_p
        i = C.c_int
        lib.oracle_decode_contig.argtypes = [i, i, i, i, C.c_double, p, i, p, p, i, p, p, p, i, i, i, i, p, i, p, p]
        lib.oracle_decode_paged.argtypes = [i, i, i, i, C.c_double, p, i, p, p, C.c_long, p, i, p, p, p, i, p, p]
        lib.oracle_gather_paged.argtypes = [i, i, i, p, p, C.c_long, p, i, i, i, i, p, p]
        lib.oracle_lse_merge.argtypes = [i, i, i, p, p, p, p]
        lib.oracle_threads.argtypes = []
        lib.oracle_set_threads.argtypes = [C.c_int]
        lib.oracle_set_threads.restype = None
        for f in (lib.oracle_decode_contig, lib.oracle_decode_paged, lib.oracle_gather_paged,
                  lib.oracle_lse_merge, lib.oracle_threads):
            f.restype = C.c_int
        _lib = lib
    return _lib


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


def threads() -> int:
    return int(_load().oracle_threads())


def set_threads(n: int) -> None:
    """Threads of the following oracle calls (OpenMP)."""
    _load().oracle_set_threads(int(n))


def decode_contig(q, prefix_k, prefix_v, suffix_k, suffix_v, suffix_len, scale: float,
                  prefix_range=None, suffix_range=None, rows=None):
    """Fork-decode attention over contiguous KV.  Returns (out [N][Hq][d], lse [N][Hq]) in fp64.

    prefix_range / suffix_range restrict the keys to [lo, hi) of the prefix / suffix
    positions; rows restricts the computed rows to ids b*Hq + h (others left NaN).
    """
    q = _c(q, np.uint16)
    pk, pv = _c(prefix_k, np.uint16), _c(prefix_v, np.uint16)
    sk, sv = _c(suffix_k, np.uint16), _c(suffix_v, np.uint16)
    sl = _c(suffix_len, np.int32)
    N, Hq, d = q.shape
    Hkv, Lp = pk.shape[0], pk.shape[1]
    cap = sk.shape[2]
    assert pk.shape == (Hkv, Lp, d) and pv.shape == pk.shape
    assert sk.shape == (N, Hkv, cap, d) and sv.shape == sk.shape and sl.shape == (N,)
    plo, phi = (0, Lp) if prefix_range is None else prefix_range
    slo, shi = (0, cap) if suffix_range is None else suffix_range
    out = np.full((N, Hq, d), np.nan)
    lse = np.full((N, Hq), np.nan)
    r = None if rows is None else _c(rows, np.int32)
    rc = _load().oracle_decode_contig(N, Hq, Hkv, d, float(scale), _ptr(q), Lp, _ptr(pk), _ptr(pv), cap,
                                      _ptr(sk), _ptr(sv), _ptr(sl), int(plo), int(phi), int(slo), int(shi),
                                      _ptr(r), 0 if r is None else len(r), _ptr(out), _ptr(lse))
    if rc == -3:
        raise ValueError("a suffix length is outside [0, suffix capacity]")
    if rc != 0:
        raise RuntimeError(f"oracle_decode_contig failed: {rc}")
    return out, lse


def decode_paged(q, k_pool, v_pool, page_table, seq_prefix_len, suffix_len, scale: float, rows=None):
    """Fork-decode attention over a paged pool.  Returns (out [S][Hq][d], lse [S][Hq]) in fp64."""
    q = _c(q, np.uint16)
    kp, vp = _c(k_pool, np.uint16), _c(v_pool, np.uint16)
    pt = _c(page_table, np.int32)
    spl, sl = _c(seq_prefix_len, np.int32), _c(suffix_len, np.int32)
    S, Hq, d = q.shape
    n_pages, Hkv, P = kp.shape[0], kp.shape[1], kp.shape[2]
    out = np.full((S, Hq, d), np.nan)
    lse = np.full((S, Hq), np.nan)
    r = None if rows is None else _c(rows, np.int32)
    rc = _load().oracle_decode_paged(S, Hq, Hkv, d, float(scale), _ptr(q), P, _ptr(kp), _ptr(vp), n_pages,
                                     _ptr(pt), pt.shape[1], _ptr(spl), _ptr(sl), _ptr(r),
                                     0 if r is None else len(r), _ptr(out), _ptr(lse))
    if rc != 0:
        raise RuntimeError(f"oracle_decode_paged failed: {rc}")
    return out, lse


def gather_paged(k_pool, v_pool, page_table, seq: int, prefix_len: int, suffix_len: int):
    """Host gather of one paged sequence into contiguous [Hkv][L][d] K and V (bit copies)."""
    kp, vp = _c(k_pool, np.uint16), _c(v_pool, np.uint16)
    pt = _c(page_table, np.int32)
    _, Hkv, P, d = kp.shape
    L = prefix_len + suffix_len
    ko = np.empty((Hkv, L, d), np.uint16)
    vo = np.empty((Hkv, L, d), np.uint16)
    rc = _load().oracle_gather_paged(Hkv, d, P, _ptr(kp), _ptr(vp), kp.shape[0], _ptr(pt), pt.shape[1], seq,
                                     prefix_len, suffix_len, _ptr(ko), _ptr(vo))
    if rc != 0:
        raise RuntimeError(f"oracle_gather_paged failed: {rc}")
    return ko, vo


def lse_merge(o_parts, lse_parts):
    """Merge per-part (o, lse) into the union's (o, lse).  o_parts [R][P][d], lse_parts [R][P] (fp64)."""
    op = _c(o_parts, np.float64)
    lp = _c(lse_parts, np.float64)
    R, P, d = op.shape
    assert lp.shape == (R, P)
    out = np.empty((R, d))
    lse = np.empty(R)
    rc = _load().oracle_lse_merge(R, P, d, _ptr(op), _ptr(lp), _ptr(out), _ptr(lse))
    if rc != 0:
        raise RuntimeError(f"oracle_lse_merge failed: {rc}")
    return out, lse


def decode_workload(w, rows=None):
    """Oracle result for a ContigWorkload or PagedWorkload at its current lengths."""
    if hasattr(w, "prefix_k"):
        return decode_contig(w.q, w.prefix_k, w.prefix_v, w.suffix_k, w.suffix_v, w.suffix_len,
                             w.spec.softmax_scale, rows=rows)
    return decode_paged(w.q, w.k_pool, w.v_pool, w.page_table, w.seq_prefix_len, w.suffix_len,
                        w.spec.softmax_scale, rows=rows)
