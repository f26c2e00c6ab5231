"""GPU parity of gmm_assign_topk (Sec. 4.2 single assignment, Sec. 4.3 multiple
assignment) against the fp64 checker: indices identical wherever the checker's
top-m margin exceeds 1e-6, responsibilities within 1e-4."""
import sys

import numpy as np
import pytest

import gmm_synth as g
import oracle
from gmmcheck import check_assign, gpu_assign

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _run(x, th, m, tau, label, min_checked=0.9):
    ref = oracle.assign_topk(x, *th, m, tau, mr=m + 1)
    gidx, gresp = gpu_assign(x, *th, m, tau)
    frac = check_assign(gidx, gresp, ref, m, tau, label, min_checked)
    kept = (gidx >= 0).sum(axis=0)
    _say(f"  {label}: checked {frac:.4f} of ranks, kept per rank {kept.tolist()}")
    return gidx, gresp


def test_tiny_trained():
    """The paper's setting: m = 2, tau = 1/K, at parameters after a few EM iterations."""
    x, th0 = g.make("tiny")
    f = oracle.fit(x, *th0, 5, keep_thetas=True)
    th = f["thetas"][-1]
    _run(x, th, 2, 1.0 / 8, "tiny m2")


@pytest.mark.parametrize("n,d,kt,k,m", [
    (1000, 37, 6, 45, 2), (3001, 128, 40, 64, 3), (2049, 200, 10, 17, 1), (777, 256, 8, 8, 8),
    (5, 3, 2, 2, 2), (1500, 150, 7, 40, 4), (20000, 8, 4, 300, 2),
    (1200, 768, 10, 70, 2), (800, 1024, 5, 16, 3), (1500, 513, 6, 20, 2),
    (5000, 64, 40, 4500, 2), (4300, 400, 12, 4200, 2), (900, 850, 6, 12, 2)])
def test_ragged_shapes(n, d, kt, k, m):
    w = g.custom(f"a{n}_{d}_{k}", n, d, kt, k, data_seed=n + d, init_seed=k + 17)
    x, (wt, mu, var) = g.make(w)
    var = np.where(var > 0, var, np.float32(1.0)).astype(np.float32)
    f = oracle.fit(x, wt, mu, var, 2, keep_thetas=True)
    _run(x, f["thetas"][-1], m, 1.0 / k, f"n{n} d{d} k{k} m{m}", min_checked=0.9)


def test_small_paper_shape():
    """N = 5000 rows of the paper-shape small workload, K = 1024, at Theta_0 and Theta_2."""
    x, th0 = g.make(g.custom("s5k", 5000, 128, 1024, 1024, data_seed=2, init_seed=1002))
    _run(x, th0, 2, 1.0 / 1024, "small Theta_0", min_checked=0.9)
    f = oracle.fit(x, *th0, 2, keep_thetas=True)
    _run(x, f["thetas"][-1], 2, 1.0 / 1024, "small Theta_2", min_checked=0.9)


def test_tau_zero_and_m_one():
    x, th0 = g.make("tiny")
    f = oracle.fit(x, *th0, 3, keep_thetas=True)
    gidx, _ = _run(x, f["thetas"][-1], 3, 0.0, "tau 0")
    gidx1, gresp1 = _run(x, f["thetas"][-1], 1, 0.5, "m 1")
    assert np.all(gidx1[:, 0] >= 0) and np.all(gresp1[:, 0] > 0)


def test_collapsed_and_dead_components():
    w = g.custom("acol", 6000, 64, 12, 40, data_seed=5, init_seed=55)
    x, (wt, mu, var) = g.make(w)
    rng = np.random.default_rng(0)
    var = var.copy()
    mu = mu.copy()
    for c in rng.choice(40, 10, replace=False):
        var[c] = rng.uniform(1e-5, 1e-3, var.shape[1]).astype(np.float32)
        mu[c] = x[rng.integers(0, x.shape[0])] + np.float32(1e-3)
    wt = wt.copy()
    wt[[3, 9]] = 0.0
    wt = (wt / wt.sum()).astype(np.float32)
    gidx, _ = _run(x, (wt, mu, var), 2, 1.0 / 40, "collapsed+dead", min_checked=0.9)
    assert not np.isin(gidx, [3, 9]).any()


def test_many_equal_candidates_take_the_exact_path():
    """Forty copies of one component (plus a few others): a point whose T = m + 2 largest
    components include a copy has all forty among its candidates, more than the collection
    pass keeps, so the exact all-component path must produce its ranking, ties going to the
    lower index, and its responsibilities to fp32 rounding."""
    w = g.custom("adup", 2000, 16, 4, 48, data_seed=9, init_seed=99)
    x, (wt, mu, var) = g.make(w)
    mu = mu.copy()
    var = var.copy()
    mu[:40] = mu[0]
    var[:40] = var[0]
    wt = np.full(48, 1.0 / 48, dtype=np.float32)
    m = 4
    _run(x, (wt, mu, var), m, 1e-4, "duplicates", min_checked=0.0)
    gidx, gresp = gpu_assign(x, wt, mu, var, m, 1e-4)
    ref = oracle.assign_topk(x, wt, mu, var, m, 1e-4, mr=m + 2)
    # exact ties among the copies: the order is fixed by the index rule, so every index matches
    np.testing.assert_array_equal(gidx, ref[0])
    exact = (ref[2] < 40).any(axis=1)
    assert exact.sum() > 100
    _say(f"  {exact.sum()} of {len(exact)} points have a copy among their {m + 2} largest")
    np.testing.assert_allclose(gresp[exact], ref[1][exact], atol=1e-6)
    np.testing.assert_allclose(gresp, ref[1], atol=1e-4)


def test_deterministic():
    x, th0 = g.make("tiny")
    a = gpu_assign(x, *th0, 2, 0.125)
    b = gpu_assign(x, *th0, 2, 0.125)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_deterministic_many_waves():
    """Bitwise identical results over repeated calls when every wave of the collection pass
    appends candidates (K = 512: four 32-component blocks per wave) and routed components
    (collapsed variances) append theirs too: the candidates are summed in a fixed order."""
    w = g.custom("adet", 20000, 96, 64, 512, data_seed=21, init_seed=2021)
    x, (wt, mu, var) = g.make(w)
    rng = np.random.default_rng(4)
    var = var.copy()
    mu = mu.copy()
    for c in rng.choice(512, 12, replace=False):
        var[c] = rng.uniform(1e-5, 1e-3, var.shape[1]).astype(np.float32)
        mu[c] = x[rng.integers(0, x.shape[0])] + np.float32(1e-3)
    th = (wt, mu, var)
    a = _run(x, th, 2, 1.0 / 512, "K=512 + routed", min_checked=0.9)
    for rep in range(4):
        b = gpu_assign(x, *th, 2, 1.0 / 512)
        assert np.array_equal(a[0], b[0]), f"indices differ on repeat {rep}"
        assert np.array_equal(a[1].view(np.uint32), b[1].view(np.uint32)), \
            f"responsibilities differ on repeat {rep}"
