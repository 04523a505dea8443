"""Shared helpers of the GPU tests (no test functions here)."""

import sys

import numpy as np

# Tolerances. bf16 I/O with fp32 accumulation: max-abs 1e-2 (relative to
# |o| where |o| > 1) and mean-abs 1e-3 against the float64 oracle, plus a per-row relative L2 bound that a
# kernel dropping a whole block cannot meet on near-uniform attention. fp32
# I/O: the only error sources are fp32 rounding and the hardware exp2, so the
# bounds are far tighter.
TOL = {
    "bf16": dict(max_abs=1e-2, mean_abs=1e-3, rel_l2=2e-2),
    "f32": dict(max_abs=1e-4, mean_abs=1e-5, rel_l2=1e-5),
}


def say(*a):
    print(*a, file=sys.stderr, flush=True)


def compare(got: np.ndarray, want: np.ndarray, out_dtype: str, rows=None, what=""):
    """Element-wise comparison of kernel output rows with oracle rows."""
    if rows is not None:
        got, want = got[rows], want[rows]
    assert got.shape == want.shape
    assert np.isfinite(want).all()
    assert np.isfinite(got).all(), f"{what}: non-finite outputs"
    tol = TOL[out_dtype]
    diff = np.abs(got - want)
    # The max-abs gate holds for outputs of magnitude up to 1 (the configured
    # workloads' outputs are far smaller). Above 1 it scales with |o|: a bf16
    # output in [4, 8) alone carries up to half an ulp = 2^-6 of rounding, so a
    # fixed 1e-2 could not be met by any bf16 kernel on the sharp inputs.
    max_abs = float((diff / np.maximum(1.0, np.abs(want))).max())
    mean_abs = float(diff.mean())
    num = np.sqrt(((got - want) ** 2).sum(axis=-1))
    den = np.sqrt((want ** 2).sum(axis=-1))
    rel = float((num / np.maximum(den, 1e-6)).max())
    say(f"  {what}: max_abs={max_abs:.3e} mean_abs={mean_abs:.3e} rel_l2={rel:.3e} n={diff.size}")
    assert max_abs <= tol["max_abs"], (what, max_abs)
    assert mean_abs <= tol["mean_abs"], (what, mean_abs)
    assert rel <= tol["rel_l2"], (what, rel)
    return max_abs, mean_abs, rel


def rows_of(batch, reqs):
    return np.concatenate([np.arange(batch.q_start[r], batch.q_start[r + 1]) for r in reqs])
