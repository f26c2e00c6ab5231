"""GPU parity on the code paths the full-size workloads take, against the fp64 checker.

The dense statistics pass sums each (64-component block, chunk of points) workgroup's
statistics on fp32 MFMA and moves the fp32 sums into fp64 every 4096 queued points.  At the
N = 1e8 workload a chunk holds 781,250 points and the busiest blocks queue far more than 4096
of them, but at the sizes the checker finishes in seconds the automatic chunking makes chunks
of about a thousand points, so the fp32 runs never reach their full length.  These tests cap
the chunk count (gmm_set_stats_chunk_limit) so that the queues of the small workload
(D = 128, k_stats_well) and of an IVF slice (D = 768, k_stats_wide) run past 4096 points:
every fp32 run then has the length it has at full size, and the fp32 -> fp64 step runs several
times per workgroup.  A numpy lower bound of the queue lengths shows that it does.

The other cases are the component counts whose code paths the ragged-shape tests miss at
D <= 128: K = 2048 (the refinement thresholds of more than 1024 components are read from
global memory instead of LDS) and K = 4160 (more than 64 blocks of 64 components: no per-point
block masks, every point enters every block, and the stored exact pairs are still left out).
"""
import sys
import time

import numpy as np
import pytest

import gmm_synth as g
import oracle
from gmmcheck import (FOLD_POINTS, check_params, check_stats, gpu_estep, gpu_mstep,
                      queue_lower_bound, to_dev)

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


class _ChunkLimit:
    """Caps the statistics pass's chunk count for the duration of a with-block."""

    def __init__(self, limit):
        self.limit = limit

    def __enter__(self):
        import paper_2606_10896_amd as gmm
        gmm.gmm_set_stats_chunk_limit(self.limit)

    def __exit__(self, *exc):
        import paper_2606_10896_amd as gmm
        gmm.gmm_set_stats_chunk_limit(0)


def _compare(x, th, label, xd=None):
    n = x.shape[0]
    ref = oracle.iterate(x, *th)
    st = gpu_estep(x, *th, xd=xd)
    r1 = check_stats(st, ref, label)
    w, mu, var = gpu_mstep(st, float(n), *th)
    r2 = check_params(w, mu, var, ref, n, label)
    _say(f"  {label}: {r1} {r2}")
    return ref


@pytest.mark.timeout(900)
def test_small_workload_one_chunk_full_fp32_runs():
    """N = 1e5, D = 128, K = 1024 with every block's points in one chunk: teacher-forced at
    Theta_0 and at the checker's Theta_3."""
    t0 = time.time()
    x, th0 = g.make("small")
    (xd,) = to_dev(x)
    qmax = queue_lower_bound(x, *th0, chunk_rows=x.shape[0])
    _say(f"  busiest block queues at least {qmax} points (fold every {FOLD_POINTS})")
    assert qmax > 2 * FOLD_POINTS
    thetas = [th0]
    th = th0
    for t in range(3):
        r = oracle.iterate(x, *th)
        th = (r["weights"].astype(np.float32), r["means"].astype(np.float32),
              r["vars"].astype(np.float32))
        thetas.append(th)
    _say(f"  checker trajectory done ({time.time() - t0:.1f}s)")
    with _ChunkLimit(1):
        for t in (0, 3):
            _compare(x, thetas[t], f"small, one chunk, t={t}", xd=xd)


@pytest.mark.timeout(900)
def test_ivf_slice_one_chunk_full_fp32_runs():
    """24,000 consecutive rows of the IVF workload (D = 768, K = 4096) in one chunk, so the
    wide statistics kernel's queues run past 4096 points: teacher-forced at the random-point
    initialisation (the workload's K init rows as means, uniform weights, the slice's
    per-dimension population variance)."""
    w = g.WORKLOADS["ivf"]
    rows = 24_000
    mix = g.Mixture(w)
    x = mix.rows(0, rows, nthreads=16)
    init = g.init_rows(w)
    means = np.concatenate([mix.rows(int(r), int(r) + 1) for r in init]).astype(np.float32)
    var = np.tile(x.astype(np.float64).var(axis=0), (w.k, 1)).astype(np.float32)
    wt = np.full(w.k, 1.0 / w.k, dtype=np.float32)
    th = (wt, means, var)
    qmax = queue_lower_bound(x, *th, chunk_rows=rows)
    _say(f"  busiest block queues at least {qmax} points (fold every {FOLD_POINTS})")
    assert qmax > FOLD_POINTS
    with _ChunkLimit(1):
        _compare(x, th, "ivf rows 0..24000, one chunk")


@pytest.mark.parametrize("n,d,kt,k", [(5000, 100, 40, 2048), (4500, 128, 64, 2048),
                                      (6000, 64, 30, 4160), (5000, 37, 25, 4160),
                                      (4200, 300, 12, 4160)])
def test_large_k_shapes(n, d, kt, k):
    """K = 2048 and K = 4160 off the tile boundaries, teacher-forced over three iterations of the
    checker's trajectory."""
    spec = g.custom(f"bigk{n}_{d}_{k}", n, d, kt, k, data_seed=n + k, init_seed=d + 3)
    x, th0 = g.make(spec)
    f = oracle.fit(x, *th0, 3, keep_thetas=True)
    (xd,) = to_dev(x)
    for t, th in enumerate(f["thetas"]):
        _compare(x, th, f"n{n} d{d} k{k} t={t}", xd=xd)
