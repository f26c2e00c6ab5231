"""Pins for the checker's k-means warm start: an independent numpy Lloyd iteration (distance
matrix, argmin, bincount means), the monotone within-cluster sum of squares, a fixed point, and
the empty-centre rule; the final mixture against per-cluster sample moments."""
import numpy as np
import pytest

import oracle


def _numpy_kmeans(x, c0, n_iters):
    x64 = x.astype(np.float64)
    c = c0.astype(np.float64)
    k = c.shape[0]
    for it in range(n_iters + 1):
        d2 = ((x64[:, None, :] - c[None, :, :]) ** 2).sum(2)
        a = d2.argmin(1)
        if it == n_iters:
            break
        for q in range(k):
            if np.any(a == q):
                c[q] = x64[a == q].mean(0).astype(np.float32)
    return c, a


def _sse(x, c, a):
    return float(((x.astype(np.float64) - c[a]) ** 2).sum())


@pytest.mark.parametrize("seed,n,d,k,it", [(0, 600, 3, 5, 4), (1, 2000, 8, 12, 6), (2, 300, 1, 4, 3)])
def test_matches_numpy_lloyd(seed, n, d, k, it):
    rng = np.random.default_rng(seed)
    x = (rng.standard_normal((n, d)) * rng.uniform(0.5, 2.0, d)).astype(np.float32)
    c0 = x[rng.choice(n, k, replace=False)]
    var0 = np.full((k, d), 0.5, np.float32)
    r = oracle.kmeans(x, c0, var0, it, var_floor=0.0)
    c, a = _numpy_kmeans(x, c0, it)
    np.testing.assert_array_equal(r["assign"], a)
    np.testing.assert_allclose(r["centres"], c, rtol=1e-6, atol=1e-6)
    # the mixture: hard-assignment moments of the last assignment
    x64 = x.astype(np.float64)
    for q in range(k):
        rows = x64[a == q]
        assert r["weights"][q] == pytest.approx(len(rows) / n, abs=1e-15)
        if len(rows):
            np.testing.assert_allclose(r["means"][q], rows.mean(0), rtol=1e-12, atol=1e-12)
            np.testing.assert_allclose(r["vars"][q], rows.var(0), rtol=1e-10, atol=1e-12)


def test_within_cluster_sum_of_squares_never_grows():
    rng = np.random.default_rng(5)
    x = (rng.standard_normal((3000, 4)) * 3).astype(np.float32)
    c0 = x[:20]
    var0 = np.ones((20, 4), np.float32)
    prev = np.inf
    for it in range(8):
        r = oracle.kmeans(x, c0, var0, it)
        sse = _sse(x, r["centres"], r["assign"])
        assert sse <= prev * (1 + 1e-12)
        prev = sse


def test_fixed_point_and_empty_centre():
    x = np.array([[0.0], [1.0], [10.0], [11.0]], dtype=np.float32)
    c0 = np.array([[0.5], [10.5], [100.0]], dtype=np.float32)    # centre 2 gets no rows
    var0 = np.array([[3.0], [3.0], [7.0]], dtype=np.float32)
    r = oracle.kmeans(x, c0, var0, 3, var_floor=0.0)
    np.testing.assert_array_equal(r["assign"], [0, 0, 1, 1])
    np.testing.assert_allclose(r["centres"], c0.astype(np.float64))
    np.testing.assert_allclose(r["weights"], [0.5, 0.5, 0.0])
    np.testing.assert_allclose(r["means"][:, 0], [0.5, 10.5, 100.0])
    np.testing.assert_allclose(r["vars"][:, 0], [0.25, 0.25, 7.0])
