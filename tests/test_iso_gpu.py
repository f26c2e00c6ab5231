"""GPU parity of the isotropic calls (the paper's own model, one variance per component)
against the checker's isotropic EM, under the same tolerances as the diagonal path
(gmmcheck.py; the variance tolerance applies to the scalar variance)."""
import sys

import numpy as np
import pytest

import gmm_synth as g
import oracle
from gmmcheck import (TOL_LL, check_params_iso, check_stats, gpu_estep_iso, gpu_fit_iso,
                      gpu_mstep_iso, to_dev)

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _iso_init(th0):
    """Isotropic start from a diagonal random-point init: the mean over d of its variances."""
    w, mu, var = th0
    return w, mu, var.astype(np.float64).mean(1).astype(np.float32)


def _teacher_forced(x, thetas, label, xd=None):
    n = x.shape[0]
    for t, th in enumerate(thetas):
        ref = oracle.iso_iterate(x, *th)
        st = gpu_estep_iso(x, *th, xd=xd)
        r1 = check_stats(st, ref, f"{label} t={t}")
        err_q = np.abs(st["q"] - ref["q"]) / np.maximum(ref["q"], 1.0)
        assert err_q.max() <= 1e-4, f"{label} t={t} Q: {err_q.max():.3e}"
        w, mu, var = gpu_mstep_iso(st, float(n), *th)
        r2 = check_params_iso(w, mu, var, ref, n, f"{label} t={t}")
        _say(f"  {label} t={t}: {r1} Q {err_q.max():.2e} {r2}")


@pytest.mark.parametrize("n,d,kt,k", [(2000, 37, 5, 7), (3000, 128, 20, 64), (1800, 150, 6, 40),
                                      (1200, 250, 6, 30), (1500, 300, 6, 20), (1000, 768, 8, 33),
                                      (1000, 450, 6, 15), (800, 1000, 5, 12)])
def test_isotropic_ragged_shapes(n, d, kt, k):
    w = g.custom(f"iso{n}_{d}", n, d, kt, k, data_seed=77 + d, init_seed=99 + k)
    x, th0 = g.make(w)
    th0 = _iso_init(th0)
    (xd,) = to_dev(x)
    ref = oracle.iso_fit(x, *th0, 3, keep_thetas=True)
    _teacher_forced(x, ref["thetas"], f"iso {n}x{d} K={k}", xd=xd)


def test_isotropic_small_workload_teacher_forced():
    x, th0 = g.make("small", nthreads=16)
    th0 = _iso_init(th0)
    (xd,) = to_dev(x)
    ref = oracle.iso_fit(x, *th0, 2, keep_thetas=True)
    _teacher_forced(x, ref["thetas"], "iso small", xd=xd)


def test_isotropic_fit_tiny_free_running():
    x, th0 = g.make("tiny")
    th0 = _iso_init(th0)
    ref = oracle.iso_fit(x, *th0, 10)
    w, mu, var, hist = gpu_fit_iso(x, *th0, 10)
    err = np.abs(hist - ref["loglik_hist"]) / np.abs(ref["loglik_hist"])
    _say("  isotropic free-running LL rel err per iteration:", np.array2string(err, precision=2))
    assert err.max() <= TOL_LL
    assert np.all(np.diff(hist) >= -1e-7 * np.abs(hist[1:]))
    np.testing.assert_allclose(mu, ref["means"], rtol=1e-3, atol=1e-3)
    np.testing.assert_allclose(var, ref["vars"], rtol=1e-3)
