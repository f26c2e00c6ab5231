"""Free-running gmm_fit at the paper-shape mid workload (N = 1e6, D = 128, K = 1024):
30 EM iterations from the random-point initialisation.  EM never lowers the
log-likelihood (in exact arithmetic); the GPU trajectory must be non-decreasing
up to the log-likelihood tolerance, and the fit must end with finite
parameters, positive variances and weights summing to one."""
import sys

import numpy as np
import pytest

import gmm_synth as g
from gmmcheck import TOL_LL, gpu_fit, to_dev

pytestmark = pytest.mark.gpu


def test_mid_workload_30_iterations_monotone():
    x, th0 = g.make("mid", nthreads=16)
    (xd,) = to_dev(x)
    print(f"  mid workload {x.shape}, fitting 30 iterations", flush=True)
    w, mu, var, hist = gpu_fit(x, *th0, 30, xd=xd)
    print("  LL:", np.array2string(hist[[0, 1, 2, 5, 10, 20, 29]], precision=9), flush=True)
    sys.stdout.flush()
    assert np.all(np.isfinite(hist))
    # non-decreasing up to rounding far below the parity tolerance
    drops = hist[1:] - hist[:-1]
    assert np.all(drops >= -0.01 * TOL_LL * np.abs(hist[1:])), drops.min()
    assert hist[-1] > hist[0]
    assert np.all(np.isfinite(mu)) and np.all(var > 0) and np.all(w >= 0)
    assert abs(float(np.sum(w, dtype=np.float64)) - 1.0) < 1e-5
