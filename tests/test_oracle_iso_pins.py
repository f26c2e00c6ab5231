"""Pins for the checker's isotropic model (the paper's Sec. 2 model: one scalar variance per
component).  Expected values come from other routes: the diagonal checker with tied variances
(pinned on its own in test_oracle_pins.py), scipy's Gaussian densities, sample moments, and
EM monotonicity."""
import numpy as np
import pytest
from scipy import stats
from scipy.special import logsumexp

import oracle


def _rng(seed):
    return np.random.default_rng(seed)


def _iso_theta(rng, k, d, spread=2.0):
    w = rng.dirichlet(np.ones(k)).astype(np.float32)
    mu = (spread * rng.standard_normal((k, d))).astype(np.float32)
    var = rng.uniform(0.3, 2.0, k).astype(np.float32)
    return w, mu, var


@pytest.mark.parametrize("seed,n,d,k", [(1, 500, 7, 4), (2, 333, 1, 3), (3, 800, 16, 6)])
def test_isotropic_equals_diagonal_with_tied_variances(seed, n, d, k):
    """The isotropic E-step is the diagonal one with var_kd = var_k: same N, S, LL, and
    Q_iso = sum_d Q_kd; the isotropic variance update is the mean over d of the diagonal one
    (sum_d sum_i r (x_d - mu_d)^2 / (D N_k))."""
    rng = _rng(seed)
    w, mu, var = _iso_theta(rng, k, d)
    x = (2.0 * rng.standard_normal((n, d))).astype(np.float32)
    tied = np.repeat(var[:, None], d, axis=1)
    a = oracle.iso_iterate(x, w, mu, var, var_floor=0.0)
    b = oracle.iterate(x, w, mu, tied, var_floor=0.0)
    np.testing.assert_allclose(a["nk"], b["nk"], rtol=1e-12)
    np.testing.assert_allclose(a["s"], b["s"], rtol=1e-11, atol=1e-11)
    np.testing.assert_allclose(a["q"], b["q"].sum(1), rtol=1e-11)
    assert a["loglik"] == pytest.approx(b["loglik"], rel=1e-12)
    np.testing.assert_allclose(a["weights"], b["weights"], rtol=1e-12)
    np.testing.assert_allclose(a["means"], b["means"], rtol=1e-11, atol=1e-12)
    np.testing.assert_allclose(a["vars"], b["vars"].mean(1), rtol=1e-10)


@pytest.mark.parametrize("d", [1, 4, 32])
def test_isotropic_single_component_closed_form(d):
    """K = 1: the mean is the sample mean, the variance is the per-dimension population
    variance averaged over the dimensions (Eq. sig), LL is a sum of univariate log-pdfs."""
    rng = _rng(10 + d)
    x = (rng.standard_normal((613, d)) * 1.3 - 0.7).astype(np.float32)
    w = np.ones(1, np.float32)
    mu0 = rng.standard_normal((1, d)).astype(np.float32)
    var0 = np.array([1.7], np.float32)
    r = oracle.iso_iterate(x, w, mu0, var0, var_floor=0.0)
    x64 = x.astype(np.float64)
    np.testing.assert_allclose(r["means"][0], x64.mean(0), rtol=1e-12, atol=1e-13)
    assert r["vars"][0] == pytest.approx(x64.var(0, ddof=0).mean(), rel=1e-10)
    ll = stats.norm.logpdf(x64, loc=mu0.astype(np.float64),
                           scale=np.sqrt(np.float64(var0[0]))).sum()
    assert r["loglik"] == pytest.approx(ll, rel=1e-12)
    assert r["q"][0] == pytest.approx((x64 ** 2).sum(), rel=1e-12)


def test_isotropic_loglik_matches_scipy_mixture_density():
    rng = _rng(21)
    w, mu, var = _iso_theta(rng, 5, 3)
    x = (rng.standard_normal((300, 3)) * 2).astype(np.float32)
    comp = np.stack([np.log(np.float64(w[c])) + stats.multivariate_normal.logpdf(
        x.astype(np.float64), mean=mu[c].astype(np.float64),
        cov=np.float64(var[c]) * np.eye(3)) for c in range(5)], axis=1)
    want = logsumexp(comp, axis=1).sum()
    got = oracle.iso_estep(x, w, mu, var)["loglik"]
    assert got == pytest.approx(want, rel=1e-12)


def test_isotropic_loglik_non_decreasing():
    rng = _rng(31)
    w, mu, var = _iso_theta(rng, 6, 5, spread=1.0)
    x = (rng.standard_normal((1500, 5)) * 2).astype(np.float32)
    hist = oracle.iso_fit(x, w, mu, var, 12)["loglik_hist"]
    assert np.all(np.diff(hist) >= -1e-9 * np.abs(hist[1:]))
    assert hist[-1] > hist[0]


def test_isotropic_estep_is_additive_over_row_splits():
    rng = _rng(41)
    w, mu, var = _iso_theta(rng, 4, 6)
    x = (rng.standard_normal((900, 6)) * 2).astype(np.float32)
    a, b, whole = (oracle.iso_estep(x[:400], w, mu, var), oracle.iso_estep(x[400:], w, mu, var),
                   oracle.iso_estep(x, w, mu, var))
    for key in ("nk", "s", "q"):
        np.testing.assert_allclose(a[key] + b[key], whole[key], rtol=1e-12, atol=1e-12)
    assert a["loglik"] + b["loglik"] == pytest.approx(whole["loglik"], rel=1e-13)
