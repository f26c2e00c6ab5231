"""The seeded input generator: Philox known answers, slice addressability, recipe shape."""
import numpy as np
import pytest

import gmm_synth as g


# Known-answer vectors published with the Random123 library for philox4x32_10
# (Salmon et al., SC'11): counter, key -> output.
KAT = [
    ([0, 0, 0, 0], [0, 0], [0x6627E8D5, 0xE169C58D, 0xBC57AC4C, 0x9B00DBD8]),
    ([0xFFFFFFFF] * 4, [0xFFFFFFFF] * 2, [0x408F276D, 0x41C83B0E, 0xA20BC7C6, 0x6D5451FD]),
    ([0x243F6A88, 0x85A308D3, 0x13198A2E, 0x03707344], [0xA4093822, 0x299F31D0],
     [0xD16CFE09, 0x94FDCCEB, 0x5001E420, 0x24126EA1]),
]


@pytest.mark.parametrize("ctr,key,want", KAT)
def test_philox_known_answers(ctr, key, want):
    assert list(g.philox4x32_10(ctr, key)) == want


def test_row_slices_are_independent():
    w = g.custom("t", 5000, 24, 5, 5)
    mix = g.Mixture(w)
    full = mix.rows(0, 5000, nthreads=3)
    for a, b in [(0, 1), (17, 333), (4999, 5000), (1234, 4321)]:
        assert np.array_equal(mix.rows(a, b, nthreads=1), full[a:b])


def test_thread_count_does_not_change_bytes_or_colstats():
    w = g.custom("t", 3000, 10, 4, 4)
    mix = g.Mixture(w)
    x1, s1, q1 = mix.rows(0, 3000, nthreads=1, want_colstats=True)
    x2, s2, q2 = mix.rows(0, 3000, nthreads=7, want_colstats=True)
    assert np.array_equal(x1, x2)
    np.testing.assert_allclose(s1, x1.astype(np.float64).sum(0), rtol=1e-12)
    np.testing.assert_allclose(q1, (x1.astype(np.float64) ** 2).sum(0), rtol=1e-12)
    np.testing.assert_allclose(s2, s1, rtol=1e-12)


def test_recipe_statistics():
    """Means ~ N(0, 4), stds ~ U[0.5, 1.5], weights Dirichlet(1), rows follow the mixture."""
    w = g.custom("t", 40000, 16, 64, 64)
    mix = g.Mixture(w)
    assert abs(mix.means.std() - 2.0) < 0.1
    assert mix.stds.min() >= 0.5 and mix.stds.max() <= 1.5
    assert abs(mix.weights.sum() - 1.0) < 1e-12 and mix.weights.min() > 0
    x, comp = mix.rows(0, w.n, want_comp=True)
    counts = np.bincount(comp, minlength=64)
    # categorical frequencies within 5 binomial sd of the weights
    sd = np.sqrt(w.n * mix.weights * (1 - mix.weights))
    assert np.all(np.abs(counts - w.n * mix.weights) < 5 * sd + 1)
    # within-component standardised residuals are ~ N(0, 1)
    z = (x - mix.means[comp]) / mix.stds[comp]
    assert abs(z.mean()) < 0.01 and abs(z.std() - 1.0) < 0.01


def test_ivf_rows_are_unit_norm():
    w = g.Workload("v", 2000, 96, 128, 64, 1, 5, 1005, normalize=True)
    x = g.Mixture(w).rows(0, 2000)
    np.testing.assert_allclose(np.linalg.norm(x.astype(np.float64), axis=1), 1.0, atol=1e-6)


def test_random_point_init():
    w = g.custom("t", 2000, 8, 6, 50)
    x, (wt, mu, var) = g.make(w)
    rows = g.init_rows(w)
    assert len(set(rows.tolist())) == 50 and rows.min() >= 0 and rows.max() < 2000
    assert np.array_equal(mu, x[rows])
    np.testing.assert_allclose(var[0], x.astype(np.float64).var(0), rtol=1e-6)
    assert np.all(var == var[0]) and np.all(wt == np.float32(1 / 50))
