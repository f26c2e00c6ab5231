"""Pins for the checker's k-means++ seeding (Arthur and Vassilvitskii 2007; the paper's
alternative initialisation, Sec. 4.5 and App. C): a numpy implementation of the D^2 inversion
(numpy's own distance sums and cumulative sum; equal choices except on rounding boundaries,
which random uniforms do not hit), the margins it reports, the exact D^2 probabilities on a
tiny set (frequencies over a fine grid of uniforms), and the special cases."""
import numpy as np
import pytest

import oracle


def _numpy_kpp(x, k, u):
    x64 = x.astype(np.float64)
    n = x.shape[0]
    idx = [min(int(u[0] * n), n - 1)]
    dist = ((x64 - x64[idx[0]]) ** 2).sum(1)
    for t in range(1, k):
        c = np.cumsum(dist)
        i = int(np.searchsorted(c, u[t] * c[-1], side="right"))
        idx.append(i)
        dist = np.minimum(dist, ((x64 - x64[i]) ** 2).sum(1))
    return np.array(idx)


@pytest.mark.parametrize("seed,n,d,k", [(0, 1000, 5, 10), (1, 9000, 3, 40), (2, 5000, 17, 64),
                                        (3, 123, 2, 123)])
def test_matches_numpy_inversion(seed, n, d, k):
    rng = np.random.default_rng(seed)
    x = (rng.standard_normal((n, d)) * rng.uniform(0.5, 3.0, d)).astype(np.float32)
    u = rng.random(k)
    idx, cen = oracle.kmeanspp(x, k, u)
    np.testing.assert_array_equal(idx, _numpy_kpp(x, k, u))
    np.testing.assert_array_equal(cen, x[idx])
    assert len(set(idx.tolist())) == k     # a chosen row has distance 0 and is never drawn again


def test_second_centre_follows_squared_distance():
    """Four points on a line, first centre fixed at 0: the second is point j with probability
    d_j^2 / sum d^2, d = (1, 2, 4) -> (1, 4, 16)/21 (D would give 1, 2, 4 / 7)."""
    x = np.array([[0.0], [1.0], [2.0], [4.0]], dtype=np.float32)
    m = 21000
    counts = np.zeros(4, dtype=int)
    for i in range(m):
        idx, _ = oracle.kmeanspp(x, 2, np.array([0.1, (i + 0.5) / m]))
        counts[idx[1]] += 1
    assert idx[0] == 0 and counts[0] == 0
    np.testing.assert_allclose(counts[1:] / m, np.array([1, 4, 16]) / 21, atol=2.0 / m)


def test_special_cases():
    rng = np.random.default_rng(7)
    x = rng.standard_normal((300, 4)).astype(np.float32)
    idx, _ = oracle.kmeanspp(x, 1, np.array([0.999]))
    assert idx[0] == 299
    # duplicated rows: once one copy is a centre, its copies have distance 0
    xd = np.repeat(x[:5], 60, axis=0)
    idx, _ = oracle.kmeanspp(xd, 5, rng.random(5))
    assert len(set((idx // 60).tolist())) == 5
    # all rows equal: the total is 0 after the first centre, later centres use floor(u N)
    xs = np.ones((50, 3), dtype=np.float32)
    idx, _ = oracle.kmeanspp(xs, 3, np.array([0.5, 0.02, 0.98]))
    np.testing.assert_array_equal(idx, [25, 1, 49])


def test_margins_locate_the_target_in_the_picked_interval():
    """margin[t] = min(target - cum[pick - 1], cum[pick] - target) / total, cum the running
    sum of D^2 at draw t, checked against numpy's cumulative sums (to rounding)."""
    rng = np.random.default_rng(11)
    x = (rng.standard_normal((2000, 6)) * 2.0).astype(np.float32)
    k = 12
    u = rng.random(k)
    idx, _, mg = oracle.kmeanspp(x, k, u, want_margin=True)
    assert mg[0] == np.inf
    x64 = x.astype(np.float64)
    dist = ((x64 - x64[idx[0]]) ** 2).sum(1)
    for t in range(1, k):
        c = np.cumsum(dist)
        target = u[t] * c[-1]
        i = idx[t]
        lo = c[i - 1] if i > 0 else 0.0
        assert lo <= target < c[i]
        want = min(target - lo, c[i] - target) / c[-1]
        assert mg[t] == pytest.approx(want, rel=1e-9, abs=1e-12)
        assert 0.0 < mg[t] <= 0.5 * dist[i] / c[-1] + 1e-15
        dist = np.minimum(dist, ((x64 - x64[i]) ** 2).sum(1))
