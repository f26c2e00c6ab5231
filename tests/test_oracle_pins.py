"""Pins for the CPU checker: closed forms, brute-force enumeration, invariants.

Nothing here retypes the checker's own formulas; every expected value comes
from a different route (a library density, an enumeration over all joint
assignments, a mathematical invariant, or the EM monotonicity theorem).
"""
import math

import numpy as np
import pytest
from scipy import stats

import gmm_synth as g
import oracle
from oracle import brute


def _rng(seed):
    return np.random.default_rng(seed)


def _theta(rng, k, d, spread=2.0):
    w = rng.dirichlet(np.ones(k)).astype(np.float32)
    mu = (spread * rng.standard_normal((k, d))).astype(np.float32)
    var = rng.uniform(0.3, 2.0, (k, d)).astype(np.float32)
    return w, mu, var


# ---------------------------------------------------------------- closed forms

@pytest.mark.parametrize("d", [1, 3, 16])
def test_single_component_is_sample_mean_and_population_variance(d):
    """K=1: every responsibility is 1, so one iteration gives the sample mean and the variance
    with divisor N (Eqs. muk, sig), and LL is the sum of Gaussian log-densities."""
    rng = _rng(d)
    x = (rng.standard_normal((777, d)) * 1.7 + 0.3).astype(np.float32)
    w = np.ones(1, np.float32)
    mu0 = rng.standard_normal((1, d)).astype(np.float32)
    var0 = rng.uniform(0.5, 2.0, (1, d)).astype(np.float32)
    r = oracle.iterate(x, w, mu0, var0, var_floor=0.0)
    x64 = x.astype(np.float64)
    np.testing.assert_allclose(r["means"][0], x64.mean(0), rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(r["vars"][0], x64.var(0, ddof=0), rtol=1e-10)
    assert r["weights"][0] == pytest.approx(1.0, abs=1e-15)
    ll = stats.norm.logpdf(x64, loc=mu0.astype(np.float64), scale=np.sqrt(var0.astype(np.float64))).sum()
    assert r["loglik"] == pytest.approx(ll, rel=1e-12)
    assert r["nk"][0] == pytest.approx(777.0, rel=1e-14)
    np.testing.assert_allclose(r["q"][0], (x64 ** 2).sum(0), rtol=1e-12)


def test_loglik_matches_scipy_mixture_density():
    """LL = sum_i log sum_k pi_k N(x_i | mu_k, diag var_k), with scipy's Gaussian log-pdf."""
    rng = _rng(5)
    w, mu, var = _theta(rng, 4, 3)
    x = (rng.standard_normal((200, 3)) * 2).astype(np.float32)
    comp = np.stack([np.log(np.float64(w[c])) + stats.multivariate_normal.logpdf(
        x.astype(np.float64), mean=mu[c].astype(np.float64), cov=np.diag(var[c].astype(np.float64)))
        for c in range(4)], axis=1)
    from scipy.special import logsumexp
    want = logsumexp(comp, axis=1)
    got = oracle.estep(x, w, mu, var, want_logz=True)
    np.testing.assert_allclose(got["logz"], want, rtol=1e-12)
    assert got["loglik"] == pytest.approx(want.sum(), rel=1e-12)
    l, lz = oracle.logdens(x, w, mu, var)
    np.testing.assert_allclose(l, comp, rtol=1e-12)


# ---------------------------------------------------------------- enumeration

@pytest.mark.parametrize("seed,n,k,d", [(0, 4, 2, 1), (1, 5, 3, 2), (2, 6, 2, 2), (3, 5, 3, 1)])
def test_enumeration_marginal_and_posteriors(seed, n, k, d):
    """Sum over all K^N joint assignments: marginal likelihood = exp(LL) and posterior
    marginals = responsibilities; the statistics are the posterior-weighted sums."""
    rng = _rng(seed)
    w, mu, var = _theta(rng, k, d, spread=1.0)
    x = (rng.standard_normal((n, d)) * 1.2).astype(np.float32)
    xl = x.astype(np.float64).tolist()
    total, post = brute.enumerate_posterior(xl, w.astype(np.float64).tolist(),
                                            mu.astype(np.float64).tolist(),
                                            var.astype(np.float64).tolist())
    st = oracle.estep(x, w, mu, var)
    assert st["loglik"] == pytest.approx(math.log(total), rel=1e-12, abs=1e-12)
    post = np.array(post)
    for i in range(n):
        one = oracle.estep(x[i:i + 1], w, mu, var)
        np.testing.assert_allclose(one["nk"], post[i], rtol=1e-10, atol=1e-14)
    x64 = x.astype(np.float64)
    np.testing.assert_allclose(st["nk"], post.sum(0), rtol=1e-10)
    np.testing.assert_allclose(st["s"], post.T @ x64, rtol=1e-10, atol=1e-13)
    np.testing.assert_allclose(st["q"], post.T @ x64 ** 2, rtol=1e-10, atol=1e-13)


def test_mstep_maximises_expected_complete_loglik():
    """For the responsibilities of Theta_t (by enumeration), Theta_{t+1} is the maximiser of the
    expected complete-data log-likelihood: random perturbations never increase it."""
    rng = _rng(11)
    n, k, d = 6, 2, 2
    w, mu, var = _theta(rng, k, d, spread=1.5)
    x = (rng.standard_normal((n, d)) * 1.5).astype(np.float32)
    xl = x.astype(np.float64).tolist()
    _, post = brute.enumerate_posterior(xl, w.astype(float).tolist(), mu.astype(float).tolist(),
                                        var.astype(float).tolist())
    r = oracle.iterate(x, w, mu, var, var_floor=0.0)
    best = brute.expected_complete_loglik(xl, post, r["weights"].tolist(), r["means"].tolist(),
                                          r["vars"].tolist())
    for t in range(300):
        eps = 10.0 ** rng.uniform(-6, -1)
        w2 = np.clip(r["weights"] * np.exp(eps * rng.standard_normal(k)), 1e-12, None)
        w2 /= w2.sum()
        mu2 = r["means"] + eps * rng.standard_normal((k, d))
        v2 = r["vars"] * np.exp(eps * rng.standard_normal((k, d)))
        val = brute.expected_complete_loglik(xl, post, w2.tolist(), mu2.tolist(), v2.tolist())
        assert val <= best + 1e-12 * abs(best)


# ---------------------------------------------------------------- invariants

def test_responsibilities_sum_to_one_and_lie_in_unit_interval():
    rng = _rng(3)
    w, mu, var = _theta(rng, 7, 5)
    x = (rng.standard_normal((50, 5)) * 3).astype(np.float32)
    for i in range(50):
        nk = oracle.estep(x[i:i + 1], w, mu, var)["nk"]
        assert abs(nk.sum() - 1.0) < 1e-14
        assert nk.min() >= 0.0 and nk.max() <= 1.0


@pytest.mark.parametrize("name", ["tiny"])
def test_loglik_non_decreasing(name):
    """EM never decreases the likelihood (Dempster, Laird & Rubin 1977).  Parameters are rounded
    to fp32 between iterations, which can cost at most ~1e-9 relative."""
    x, th = g.make(name)
    f = oracle.fit(x, *th, 10)
    h = f["loglik_hist"]
    assert np.all(np.diff(h) >= -1e-9 * np.abs(h[1:]))
    assert h[-1] > h[0]


def test_loglik_non_decreasing_many_components():
    w = g.custom("c", 3000, 6, 12, 20, data_seed=21, init_seed=121)
    x, th = g.make(w)
    h = oracle.fit(x, *th, 15)["loglik_hist"]
    assert np.all(np.diff(h) >= -1e-9 * np.abs(h[1:]))


def test_affine_equivariance():
    """x -> a*x + b maps mu -> a*mu + b, var -> a^2 var and shifts LL by -N sum_d log|a_d|."""
    rng = _rng(8)
    k, d, n = 3, 4, 400
    w, mu, var = _theta(rng, k, d)
    x = (rng.standard_normal((n, d)) * 2).astype(np.float32)
    a = np.array([2.0, 0.5, 4.0, 0.25], np.float32)   # powers of two: scaling is exact
    b = np.zeros(d, np.float32)
    r0 = oracle.iterate(x, w, mu, var, var_floor=0.0)
    r1 = oracle.iterate(x * a + b, w, mu * a + b, var * a * a, var_floor=0.0)
    np.testing.assert_allclose(r1["means"], r0["means"] * a + b, rtol=1e-12, atol=1e-14)
    np.testing.assert_allclose(r1["vars"], r0["vars"] * a.astype(float) ** 2, rtol=1e-11)
    np.testing.assert_allclose(r1["weights"], r0["weights"], rtol=1e-12)
    assert r1["loglik"] == pytest.approx(r0["loglik"] - n * np.log(a.astype(float)).sum(), rel=1e-12)
    # general shift (not exact in fp32): equal to rounding
    b = np.array([3.0, -1.5, 0.25, 7.0], np.float32)
    xs = x + b
    r2 = oracle.iterate(xs, w, mu + b, var, var_floor=0.0)
    np.testing.assert_allclose(r2["means"], r0["means"] + b, rtol=1e-6, atol=1e-6)
    np.testing.assert_allclose(r2["vars"], r0["vars"], rtol=1e-5)


def test_permutation_equivariance():
    rng = _rng(9)
    w, mu, var = _theta(rng, 6, 3)
    x = (rng.standard_normal((300, 3)) * 2).astype(np.float32)
    p = rng.permutation(6)
    r0 = oracle.iterate(x, w, mu, var)
    r1 = oracle.iterate(x, w[p], mu[p], var[p])
    np.testing.assert_allclose(r1["means"], r0["means"][p], rtol=1e-12)
    np.testing.assert_allclose(r1["vars"], r0["vars"][p], rtol=1e-11)
    np.testing.assert_allclose(r1["weights"], r0["weights"][p], rtol=1e-12)
    assert r1["loglik"] == pytest.approx(r0["loglik"], rel=1e-13)


def test_duplicated_component_changes_nothing():
    """Splitting a component into two identical halves with half the weight leaves the mixture
    density, hence LL, unchanged; both halves move like the original."""
    rng = _rng(10)
    w, mu, var = _theta(rng, 4, 3)
    x = (rng.standard_normal((300, 3)) * 2).astype(np.float32)
    j = 2
    w2 = np.concatenate([w, w[j:j + 1]]); w2[j] /= 2; w2[-1] /= 2
    mu2 = np.concatenate([mu, mu[j:j + 1]]); var2 = np.concatenate([var, var[j:j + 1]])
    r0 = oracle.iterate(x, w, mu, var)
    r1 = oracle.iterate(x, w2, mu2, var2)
    assert r1["loglik"] == pytest.approx(r0["loglik"], rel=1e-12)
    for c in (j, 4):
        np.testing.assert_allclose(r1["means"][c], r0["means"][j], rtol=1e-11)
        np.testing.assert_allclose(r1["vars"][c], r0["vars"][j], rtol=1e-10)
        assert r1["weights"][c] == pytest.approx(r0["weights"][j] / 2, rel=1e-11)


def test_additivity_over_row_splits():
    x, th = g.make("tiny")
    full = oracle.estep(x, *th)
    a = oracle.estep(x[:3333], *th)
    b = oracle.estep(x[3333:], *th)
    np.testing.assert_allclose(a["nk"] + b["nk"], full["nk"], rtol=1e-12)
    np.testing.assert_allclose(a["s"] + b["s"], full["s"], rtol=1e-11, atol=1e-9)
    np.testing.assert_allclose(a["q"] + b["q"], full["q"], rtol=1e-12)
    assert a["loglik"] + b["loglik"] == pytest.approx(full["loglik"], rel=1e-13)


def test_dead_component_rule():
    """pi_k = 0: log-density -inf, N_k = 0, parameters kept, weight stays 0; the other
    components behave as in the mixture without it."""
    rng = _rng(12)
    w, mu, var = _theta(rng, 5, 3)
    x = (rng.standard_normal((200, 3)) * 2).astype(np.float32)
    w0 = w.copy(); w0[1] = 0.0
    r = oracle.iterate(x, w0, mu, var)
    assert r["weights"][1] == 0.0 and r["nk"][1] == 0.0
    assert np.array_equal(r["means"][1], mu[1].astype(np.float64))
    assert np.array_equal(r["vars"][1], var[1].astype(np.float64))
    keep = [0, 2, 3, 4]
    r2 = oracle.iterate(x, w0[keep], mu[keep], var[keep])
    assert r["loglik"] == pytest.approx(r2["loglik"], rel=1e-13)
    np.testing.assert_allclose(r["means"][keep], r2["means"], rtol=1e-12)


def test_variance_floor():
    x = np.zeros((50, 2), np.float32)
    x[:, 1] = np.linspace(-1, 1, 50)
    r = oracle.iterate(x, np.ones(1, np.float32), np.zeros((1, 2), np.float32),
                       np.ones((1, 2), np.float32), var_floor=1e-3)
    assert r["vars"][0, 0] == 1e-3
    assert r["vars"][0, 1] == pytest.approx(x[:, 1].astype(np.float64).var(), rel=1e-12)


def test_parameter_recovery_well_separated():
    """A well-separated mixture started near the truth is recovered: matched means within
    5 sd of the sampling error, weights within 5 binomial sd."""
    w = g.Workload("rec", 20000, 8, 5, 5, 1, 31, 131, mean_std=10.0)
    mix = g.Mixture(w)
    x, comp = mix.rows(0, w.n, want_comp=True)
    rng = _rng(31)
    mu0 = (mix.means + 0.5 * rng.standard_normal(mix.means.shape)).astype(np.float32)
    f = oracle.fit(x, np.full(5, 0.2, np.float32), mu0, np.ones((5, 8), np.float32), 25)
    counts = np.bincount(comp, minlength=5)
    for c in range(5):
        se = mix.stds[c] / np.sqrt(max(counts[c], 1))
        assert np.all(np.abs(f["means"][c] - mix.means[c]) < 5 * se + 1e-6)
        sd = np.sqrt(w.n * mix.weights[c] * (1 - mix.weights[c])) / w.n
        assert abs(f["weights"][c] - mix.weights[c]) < 5 * sd
        # sample variance of the component's own points (population form)
        pts = x[comp == c].astype(np.float64)
        np.testing.assert_allclose(f["vars"][c], pts.var(0), rtol=0.02)


# ---------------------------------------------------------------- top-m assignment

def _brute_rank(x, w, mu, var):
    """Per point: components sorted by log(pi_k N(x|k)) descending, ties to the lower index,
    with responsibilities, using the textbook density."""
    out = []
    for xi in x.astype(np.float64):
        lp = [math.log(w[c]) + math.log(brute.gauss_pdf_diag(xi, mu[c], var[c])) for c in range(len(w))]
        mx = max(lp)
        z = mx + math.log(sum(math.exp(v - mx) for v in lp))
        order = sorted(range(len(w)), key=lambda c: (-lp[c], c))
        out.append([(c, math.exp(lp[c] - z)) for c in order])
    return out


def test_topk_matches_brute_force_sort():
    rng = _rng(13)
    k, d = 5, 2
    w, mu, var = _theta(rng, k, d, spread=1.0)
    x = (rng.standard_normal((40, d)) * 1.5).astype(np.float32)
    ranks = _brute_rank(x, w.astype(float), mu.astype(float), var.astype(float))
    tau = 0.2
    idx, resp, ridx, rresp = oracle.assign_topk(x, w, mu, var, m=3, tau=tau, mr=4)
    kept_any_drop = False
    for i, rk in enumerate(ranks):
        assert list(ridx[i]) == [c for c, _ in rk[:4]]
        np.testing.assert_allclose(rresp[i], [r for _, r in rk[:4]], rtol=1e-12)
        for j in range(3):
            c, r = rk[j]
            if j == 0 or r > tau:
                assert idx[i, j] == c and resp[i, j] == np.float32(r)
            else:
                assert idx[i, j] == -1 and resp[i, j] == 0.0
                kept_any_drop = True
    assert kept_any_drop


def test_topk_ties_go_to_lower_index():
    w = np.array([0.25, 0.25, 0.25, 0.25], np.float32)
    mu = np.array([[0.0], [1.0], [0.0], [1.0]], np.float32)
    var = np.ones((4, 1), np.float32)
    x = np.array([[0.2], [0.9], [0.5]], np.float32)
    idx, resp = oracle.assign_topk(x, w, mu, var, m=2, tau=0.0)
    assert idx[0].tolist() == [0, 2]
    assert idx[1].tolist() == [1, 3]
    assert idx[2].tolist() == [0, 1]  # exact tie between the two distinct means


def test_topk_first_rank_always_kept():
    rng = _rng(14)
    w, mu, var = _theta(rng, 8, 3)
    x = (rng.standard_normal((30, 3)) * 2).astype(np.float32)
    idx, resp = oracle.assign_topk(x, w, mu, var, m=2, tau=1.0)  # nothing passes r > 1
    assert np.all(idx[:, 0] >= 0) and np.all(idx[:, 1] == -1) and np.all(resp[:, 1] == 0)
