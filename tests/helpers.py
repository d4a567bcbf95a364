"""Shared test helpers: tolerances, comparisons and the oracle spec of a workload."""
import numpy as np

import oracle
from oracle.layer import Spec

# tolerance on activations: max|gpu - ref| / max|ref| per tensor
TOL = {"bf16": 2e-2, "f32": 1e-5}


def spec_of(w, mode=None):
    return Spec(w.n_heads, w.n_kv_heads, w.head_dim, w.block_size, w.top_k, mode or w.mode, w.dtype,
                w.rope_base, w.rms_eps)


def rel_err(got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = float(np.max(np.abs(ref))) if ref.size else 0.0
    if ref.size == 0:
        return 0.0
    return float(np.max(np.abs(got - ref))) / (den if den > 0 else 1.0)


def assert_close(got, ref, dtype, what="", tol=None):
    tol = TOL[dtype] if tol is None else tol
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    assert np.all(np.isfinite(got)), f"{what}: non-finite values"
    e = rel_err(got, ref)
    assert e <= tol, f"{what}: rel err {e:.3e} > {tol:.1e}"
    return e


def assert_close_with_infs(got, ref, dtype, what="", tol=None):
    """Infinite entries must coincide exactly; finite ones within tolerance."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    gi, ri = ~np.isfinite(got), ~np.isfinite(ref)
    assert np.array_equal(gi, ri), f"{what}: infinite entries differ ({int((gi != ri).sum())})"
    assert np.array_equal(got[gi], ref[ri]), f"{what}: signs of infinities differ"
    if np.any(~ri):
        return assert_close(got[~gi], ref[~ri], dtype, what, tol)
    return 0.0


def f64(a):
    return np.asarray(a, dtype=np.float64)
