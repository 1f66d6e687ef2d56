"""Shared helpers of the GPU parity tests (comparison rules, sampling)."""
import numpy as np

# Floating-point bar: the layer output may differ from the oracle's exact
# (double precision) value by at most 1e-5 of the mass of the summed terms,
# sum_j |Ã_ij ζ_jk| + |b_k|, the scale that bounds fp32 summation error.
TOL = 1e-5


def mass_error(got, z, m, relu=False):
    """max |got - act(z)| / m, with m == 0 requiring an exact zero."""
    ref = np.maximum(z, 0.0) if relu else z
    got = np.asarray(got, dtype=np.float64)
    diff = np.abs(got - ref)
    zero = m == 0
    if np.any(zero) and np.any(diff[zero] != 0):
        return np.inf
    m = np.where(zero, 1.0, m)
    return float((diff / m).max()) if diff.size else 0.0


def plain_rel_error(got, z, m):
    """max relative error over entries whose value is not a near-cancellation
    (|z| >= 1e-3 m); reported, not gated."""
    sel = np.abs(z) >= 1e-3 * m
    if not np.any(sel):
        return 0.0
    return float((np.abs(np.asarray(got, np.float64)[sel] - z[sel]) / np.abs(z[sel])).max())


def u64(t):
    """numpy uint64 view of an int64 torch tensor of packed words."""
    return t.cpu().numpy().view(np.uint64)


def sample_rows(g, k, seed, extra_top=3):
    """k random rows plus the first, the last and the highest-degree rows."""
    rng = np.random.default_rng(seed)
    deg = np.diff(g.rowptr)
    top = np.argsort(deg)[-extra_top:]
    ids = np.concatenate([[0, g.n - 1], top, rng.choice(g.n, size=min(k, g.n), replace=False)])
    return np.unique(ids).astype(np.int64)
