"""GPU parity of the reduced-precision calls (gmm_estep_accumulate_screened,
gmm_fit_screened) against the fp64 checker, under their own tolerances
(SCREENED_TOL in gmmcheck.py, stated in the C header).

These calls keep the screening pass's log-densities (split bf16 products,
fp32 accumulation) for the pairs that the exact calls recompute in the direct
form; every other part of the E-step is shared.  So the tests check the
looser tolerances against the checker, that the screened statistics stay
within them of the exact call's, that the fit is the screened E-step followed
by the M-step, and that the call is deterministic.
"""
import sys

import numpy as np
import pytest

import gmm_synth as g
import oracle
from gmmcheck import (SCREENED_TOL, check_params, check_stats, gpu_estep, gpu_fit, gpu_mstep,
                      to_dev)

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _teacher_forced(x, thetas, label, xd=None):
    n = x.shape[0]
    for t, th in enumerate(thetas):
        ref = oracle.iterate(x, *th)
        st = gpu_estep(x, *th, xd=xd, screened=True)
        r1 = check_stats(st, ref, f"{label} t={t}", tol=SCREENED_TOL)
        w, mu, var = gpu_mstep(st, float(n), *th)
        r2 = check_params(w, mu, var, ref, n, f"{label} t={t}", tol=SCREENED_TOL)
        _say(f"  screened {label} t={t}: {r1} {r2}")


def test_tiny_teacher_forced_all_iterations():
    x, th0 = g.make("tiny")
    f = oracle.fit(x, *th0, 10, keep_thetas=True)
    _teacher_forced(x, f["thetas"], "tiny")


@pytest.mark.parametrize("n,d,kt,k", [
    (63, 16, 3, 5), (1000, 37, 6, 45), (3001, 128, 40, 64), (2049, 200, 10, 17),
    (20000, 8, 4, 300), (2000, 300, 8, 24), (1200, 768, 10, 70)])
def test_ragged_shapes(n, d, kt, k):
    """Ragged points, dimensions and components: split-bf16 screening from the split tile
    (d <= 128) and split on the fly (d > 256), fp32 screening (d = 200)."""
    w = g.custom(f"r{n}_{d}_{k}", n, d, kt, k, data_seed=n + d, init_seed=k + 17)
    x, (wt, mu, var) = g.make(w)
    var = np.where(var > 0, var, np.float32(1.0)).astype(np.float32)
    f = oracle.fit(x, wt, mu, var, 3, keep_thetas=True)
    _teacher_forced(x, f["thetas"], f"n{n} d{d} k{k}")


def test_small_teacher_forced():
    """Paper-shape small (N=1e5, D=128, K=1024) at Theta_0 and Theta_2 of the checker's
    trajectory."""
    x, th0 = g.make("small")
    (xd,) = to_dev(x)
    th = th0
    thetas = [th0]
    for t in range(2):
        r = oracle.iterate(x, *th)
        th = (r["weights"].astype(np.float32), r["means"].astype(np.float32),
              r["vars"].astype(np.float32))
        thetas.append(th)
    _teacher_forced(x, [thetas[0], thetas[2]], "small", xd=xd)


def test_collapsed_components():
    """Near-floor variances: those components are ill-conditioned and take the direct form in
    both calls, so the screened call still meets its tolerances."""
    w = g.custom("col", 6000, 64, 12, 40, data_seed=5, init_seed=55)
    x, (wt, mu, var) = g.make(w)
    rng = np.random.default_rng(0)
    var = var.copy()
    for c in rng.choice(40, 10, replace=False):
        var[c] = rng.uniform(1e-5, 1e-3, var.shape[1]).astype(np.float32)
        mu[c] = x[rng.integers(0, x.shape[0])] + np.float32(1e-3)
    _teacher_forced(x, [(wt, mu, var)], "collapsed")


def test_screened_close_to_exact():
    """The screened statistics against the exact call's on the same input (a tighter view of
    the same error than the checker comparison: both share the dense part)."""
    x, th0 = g.make("tiny")
    f = oracle.fit(x, *th0, 5, keep_thetas=True)
    for t in (0, 4):
        a = gpu_estep(x, *f["thetas"][t])
        b = gpu_estep(x, *f["thetas"][t], screened=True)
        en = np.abs(a["nk"] - b["nk"]) / np.maximum(a["nk"], 1.0)
        ell = abs(a["loglik"] - b["loglik"]) / abs(a["loglik"])
        _say(f"  t={t}: screened vs exact N_k {en.max():.2e} LL {ell:.2e}")
        assert en.max() <= SCREENED_TOL["n"] and ell <= SCREENED_TOL["ll"]


def test_fit_is_screened_estep_then_mstep():
    """gmm_fit_screened over 3 iterations equals 3 rounds of the screened E-step and the
    M-step, bit for bit, and its log-likelihoods are the E-steps' ones."""
    x, th0 = g.make("tiny")
    n = x.shape[0]
    w, mu, var, hist = gpu_fit(x, *th0, 3, screened=True)
    th = th0
    lls = []
    for _ in range(3):
        st = gpu_estep(x, *th, screened=True)
        lls.append(st["loglik"])
        th = gpu_mstep(st, float(n), *th)
    for u, v in zip((w, mu, var), th):
        assert np.array_equal(u, v)
    assert np.array_equal(hist, np.array(lls))


def test_fit_free_running_against_checker():
    x, th0 = g.make("tiny")
    ref = oracle.fit(x, *th0, 10)
    w, mu, var, hist = gpu_fit(x, *th0, 10, screened=True)
    err = np.abs(hist - ref["loglik_hist"]) / np.abs(ref["loglik_hist"])
    _say("  screened free-running LL rel err per iteration:", np.array2string(err, precision=2))
    assert err.max() <= SCREENED_TOL["ll"]
    np.testing.assert_allclose(mu, ref["means"], rtol=1e-3, atol=1e-3)


def test_bitwise_deterministic():
    x, th0 = g.make("tiny")
    a = gpu_estep(x, *th0, screened=True)
    b = gpu_estep(x, *th0, screened=True)
    for key in ("nk", "s", "q"):
        assert np.array_equal(a[key], b[key])
    assert a["loglik"] == b["loglik"]
