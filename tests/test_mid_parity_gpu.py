"""GPU parity at the paper-shape mid workload (N = 1e6, D = 128, K = 1024; the paper's Table 1
row N = 1M), against the fp64 checker on all 1e6 points.

Teacher-forced at the random-point initialisation Theta_0 and at the checker's Theta_3, where
components have started to narrow onto groups of points.  Each is checked twice: with the
library's own chunking of the dense statistics pass (128 chunks of 7,813 points) and with 16
chunks of 62,500 points, whose busiest blocks queue well over 4096 points, so that the fp32
runs of the dense statistics reach the length they have at N = 1e8."""
import sys
import time

import numpy as np
import pytest

import gmm_synth as g
import oracle
from gmmcheck import check_params, check_stats, gpu_estep, gpu_mstep, to_dev

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.mark.timeout(1100)
def test_mid_workload_teacher_forced():
    import paper_2606_10896_amd as gmm
    t0 = time.time()
    x, th0 = g.make("mid", nthreads=16)
    (xd,) = to_dev(x)
    n = x.shape[0]
    _say(f"  mid workload {x.shape} ready ({time.time() - t0:.1f}s)")
    refs = {}
    th = th0
    thetas = {0: th0}
    for t in range(4):
        r = oracle.iterate(x, *th)
        if t in (0, 3):
            refs[t] = r
        th = (r["weights"].astype(np.float32), r["means"].astype(np.float32),
              r["vars"].astype(np.float32))
        if t < 3:
            thetas[t + 1] = th
        _say(f"  checker iteration {t} done ({time.time() - t0:.1f}s)")
    try:
        for limit in (0, 16):
            gmm.gmm_set_stats_chunk_limit(limit)
            for t in (0, 3):
                label = f"mid t={t} chunks={'auto' if limit == 0 else limit}"
                st = gpu_estep(x, *thetas[t], xd=xd)
                r1 = check_stats(st, refs[t], label)
                w, mu, var = gpu_mstep(st, float(n), *thetas[t])
                r2 = check_params(w, mu, var, refs[t], n, label)
                _say(f"  {label}: {r1} {r2}")
    finally:
        gmm.gmm_set_stats_chunk_limit(0)
