"""GPU parity: the HIP path through the C ABI against the fp64 CPU checker.

Teacher-forced: both sides receive the same fp32 parameters Theta_t (taken
from the checker's own trajectory), and the GPU statistics, log-likelihood
and M-step are compared under the tolerances in gmmcheck.py.
"""
import sys
import time

import numpy as np
import pytest

import gmm_synth as g
import oracle
from gmmcheck import (check_params, check_stats, gpu_estep, gpu_fit, gpu_mstep, to_dev,
                      TOL_LL)

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _teacher_forced(x, thetas, label, xd=None):
    n = x.shape[0]
    for t, th in enumerate(thetas):
        ref = oracle.iterate(x, *th)
        st = gpu_estep(x, *th, xd=xd)
        r1 = check_stats(st, ref, f"{label} t={t}")
        w, mu, var = gpu_mstep(st, float(n), *th)
        r2 = check_params(w, mu, var, ref, n, f"{label} t={t}")
        _say(f"  {label} t={t}: {r1} {r2}")


def test_tiny_teacher_forced_all_iterations():
    x, th0 = g.make("tiny")
    f = oracle.fit(x, *th0, 10, keep_thetas=True)
    _teacher_forced(x, f["thetas"], "tiny")


@pytest.mark.parametrize("n,d,kt,k", [
    (1, 16, 3, 1), (5, 3, 2, 2), (63, 16, 3, 5), (1000, 37, 6, 45), (5000, 100, 20, 33),
    (3001, 128, 40, 64), (2049, 200, 10, 17), (777, 256, 8, 8), (4000, 64, 5, 1),
    (20000, 8, 4, 300), (1500, 150, 7, 40),
    # wide D: 32-point screening tiles, dimensions split over the statistics waves
    (2000, 300, 8, 24), (1500, 513, 6, 20), (1200, 768, 10, 70), (800, 1024, 5, 16),
    (2500, 640, 12, 33), (900, 1000, 4, 9), (1800, 450, 9, 28), (1000, 850, 6, 20)])
def test_ragged_shapes(n, d, kt, k):
    """Shapes off every tile boundary: points, dimensions and components."""
    w = g.custom(f"r{n}_{d}_{k}", n, d, kt, max(k, 1), data_seed=n + d, init_seed=k + 17)
    if n < k:
        pytest.skip("random-point init needs n >= k")
    x, (wt, mu, var) = g.make(w)
    # a single point has zero population variance: start such fits from unit variances
    var = np.where(var > 0, var, np.float32(1.0)).astype(np.float32)
    f = oracle.fit(x, wt, mu, var, 3, keep_thetas=True)
    _teacher_forced(x, f["thetas"], f"n{n} d{d} k{k}")


def test_small_teacher_forced():
    """Paper-shape small (N=1e5, D=128, K=1024) at Theta_0 and at Theta_3 of the checker's
    trajectory, where components have started to collapse onto single points."""
    t0 = time.time()
    x, th0 = g.make("small")
    (xd,) = to_dev(x)
    th = th0
    thetas = [th0]
    for t in range(3):
        r = oracle.iterate(x, *th)
        th = (r["weights"].astype(np.float32), r["means"].astype(np.float32),
              r["vars"].astype(np.float32))
        thetas.append(th)
        _say(f"  checker iteration {t} done ({time.time() - t0:.1f}s)")
    _teacher_forced(x, [thetas[0], thetas[3]], "small", xd=xd)


def test_collapsed_components_use_the_exact_path():
    """Components with variances near the floor (and far from the origin) are hopeless for the
    fp32 expanded form; the GPU must still match the checker."""
    w = g.custom("col", 6000, 64, 12, 40, data_seed=5, init_seed=55)
    x, (wt, mu, var) = g.make(w)
    rng = np.random.default_rng(0)
    var = var.copy()
    for c in rng.choice(40, 10, replace=False):
        var[c] = rng.uniform(1e-5, 1e-3, var.shape[1]).astype(np.float32)
        mu[c] = x[rng.integers(0, x.shape[0])] + np.float32(1e-3)
    _teacher_forced(x, [(wt, mu, var)], "collapsed")


def test_dead_components():
    w = g.custom("dead", 3000, 24, 6, 10, data_seed=3, init_seed=33)
    x, (wt, mu, var) = g.make(w)
    wt = wt.copy()
    wt[[1, 7]] = 0.0
    wt /= wt.sum()
    wt = wt.astype(np.float32)
    ref = oracle.iterate(x, wt, mu, var)
    st = gpu_estep(x, wt, mu, var)
    assert st["nk"][1] == 0.0 and st["nk"][7] == 0.0
    check_stats(st, ref, "dead")
    w2, mu2, var2 = gpu_mstep(st, float(x.shape[0]), wt, mu, var)
    assert w2[1] == 0.0 and np.array_equal(mu2[1], mu[1]) and np.array_equal(var2[7], var[7])
    check_params(w2, mu2, var2, ref, x.shape[0], "dead")


def test_bitwise_deterministic():
    x, th0 = g.make("tiny")
    f = oracle.fit(x, *th0, 4, keep_thetas=True)
    a = gpu_estep(x, *f["thetas"][3])
    b = gpu_estep(x, *f["thetas"][3])
    for key in ("nk", "s", "q"):
        assert np.array_equal(a[key], b[key])
    assert a["loglik"] == b["loglik"]


def test_accumulate_is_additive_over_row_chunks():
    """estep(X) equals estep(X[:a]) + estep(X[a:]): the semantics that streaming and sharding
    rely on."""
    x, th0 = g.make("tiny")
    whole = gpu_estep(x, *th0)
    a = gpu_estep(x[:3700], *th0)
    b = gpu_estep(x[3700:], *th0)
    np.testing.assert_allclose(a["nk"] + b["nk"], whole["nk"], rtol=1e-6)
    np.testing.assert_allclose(a["s"] + b["s"], whole["s"], rtol=1e-6, atol=1e-6)
    np.testing.assert_allclose(a["q"] + b["q"], whole["q"], rtol=1e-6)
    assert a["loglik"] + b["loglik"] == pytest.approx(whole["loglik"], rel=1e-9)


def test_fit_tiny_free_running():
    """gmm_fit over 10 iterations against the checker's trajectory from the same Theta_0."""
    x, th0 = g.make("tiny")
    ref = oracle.fit(x, *th0, 10)
    w, mu, var, hist = gpu_fit(x, *th0, 10)
    err = np.abs(hist - ref["loglik_hist"]) / np.abs(ref["loglik_hist"])
    _say("  free-running LL rel err per iteration:", np.array2string(err, precision=2))
    assert err.max() <= TOL_LL
    assert np.all(np.diff(hist) >= -1e-7 * np.abs(hist[1:]))
    np.testing.assert_allclose(mu, ref["means"], rtol=1e-3, atol=1e-3)


def test_fit_resume_is_bitwise():
    x, th0 = g.make("tiny")
    a = gpu_fit(x, *th0, 6)
    b1 = gpu_fit(x, *th0, 3)
    b2 = gpu_fit(x, *b1[:3], 3)
    for u, v in zip(a[:3], b2[:3]):
        assert np.array_equal(u, v)
    assert np.array_equal(a[3], np.concatenate([b1[3], b2[3]]))
