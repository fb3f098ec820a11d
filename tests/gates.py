"""Tolerance gates for comparing a computed attention output against the oracle.

Bar for floating-point outputs (bf16 inputs, fp32 accumulation):
  gate 1: max_i |x_i - o_i|                       <= 2e-3
  gate 2: max_i |x_i - o_i| / max(|o_i|, rms(o))  <= 1e-2
rms(o) is the root-mean-square of the whole oracle output, so the relative error is
floored at the typical output magnitude: an elementwise |x-o|/|o| is meaningless
where o crosses zero.  The log-sum-exp outputs are held to |x - o| <= 2e-3.
"""
import numpy as np

MAX_ABS = 2e-3
MAX_REL = 1e-2
LSE_ABS = 2e-3


def metrics(x, o) -> dict:
    x = np.asarray(x, np.float64)
    o = np.asarray(o, np.float64)
    assert x.shape == o.shape, (x.shape, o.shape)
    err = np.abs(x - o)
    rms = float(np.sqrt(np.mean(o * o))) if o.size else 0.0
    floor = np.maximum(np.abs(o), rms if rms > 0 else 1e-30)
    return {
        "max_abs": float(err.max()) if err.size else 0.0,
        "max_rel": float((err / floor).max()) if err.size else 0.0,
        "normwise": float(np.linalg.norm(x - o) / max(np.linalg.norm(o), 1e-300)) if o.size else 0.0,
        "rms": rms,
        "finite": bool(np.all(np.isfinite(x))),
    }


def passes(x, o, max_abs=MAX_ABS, max_rel=MAX_REL) -> bool:
    m = metrics(x, o)
    return m["finite"] and m["max_abs"] <= max_abs and m["max_rel"] <= max_rel


def assert_gates(x, o, what="", max_abs=MAX_ABS, max_rel=MAX_REL):
    m = metrics(x, o)
    assert m["finite"], f"{what}: non-finite values in result"
    assert m["max_abs"] <= max_abs and m["max_rel"] <= max_rel, f"{what}: gates failed {m}"
    return m


def assert_lse(x, o, what="", tol=LSE_ABS):
    x = np.asarray(x, np.float64)
    o = np.asarray(o, np.float64)
    both_inf = np.isneginf(x) & np.isneginf(o)
    assert np.array_equal(np.isneginf(x), np.isneginf(o)), f"{what}: -inf pattern differs"
    d = np.abs(np.where(both_inf, 0.0, x - o))
    assert np.all(np.isfinite(d)) and d.max(initial=0.0) <= tol, f"{what}: lse max err {d.max(initial=0.0)}"
