"""Shared test helpers: seeded inputs as float64 and the tolerance rule."""

import numpy as np

from synthetic import storage_to_f64
from synthetic import workloads as W

# Tolerance per storage dtype.
TOL = {"f32": 1e-5, "f16": 2e-2, "bf16": 3e-2}


def inputs_f64(workload, dtype=None, **shape):
    dtype = dtype or W.DEFAULT_DTYPE[workload]
    specs = W.specs(workload, dtype=dtype, **shape)
    raw = W.make_inputs(specs)
    return raw, {k: storage_to_f64(v, dtype) for k, v in raw.items()}


def close(got, ref, tol):
    """Elementwise |g - r| <= tol*|r| + tol*max|r| (a relative bound per element
    plus an absolute one scaled by the output's largest magnitude); returns
    (ok, max_abs, normwise_rel) with normwise_rel = max|g - r| / max|r|."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    scale = float(np.max(np.abs(ref))) if ref.size else 0.0
    err = np.abs(got - ref)
    ok = bool(np.all(err <= tol * np.abs(ref) + tol * scale)) and bool(np.all(np.isfinite(got)))
    mx = float(err.max()) if err.size else 0.0
    return ok, mx, (mx / scale if scale > 0 else mx)


def close_elementwise(got, ref, rtol, atol):
    """The stricter rule |g - r| <= rtol*|r| + atol with a fixed absolute floor
    (not scaled by the output's maximum); returns (ok, max_abs, max_rel), where
    max_rel is taken over the elements with |r| > atol / rtol (where the
    relative term dominates)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    err = np.abs(got - ref)
    ok = bool(np.all(err <= rtol * np.abs(ref) + atol)) and bool(np.all(np.isfinite(got)))
    big = np.abs(ref) > atol / rtol
    rel = float(np.max(err[big] / np.abs(ref[big]))) if np.any(big) else 0.0
    return ok, (float(err.max()) if err.size else 0.0), rel
