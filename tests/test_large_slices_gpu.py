"""The N = 1e8, D = 128, K = 1024 workload on three row slices (start, middle and end of
the data set; each generated on its own, the generator is row-addressable): teacher-forced
statistics against the fp64 checker, and additivity of the slice statistics.  The
parameters are K rows of the workload (its random-point initialisation rows) as means,
uniform weights and the per-dimension population variance of the union of the slices (the
full-N column statistics would need all 1e8 rows)."""
import numpy as np
import pytest

import gmm_synth as g
import oracle
from gmmcheck import check_params, check_stats, gpu_estep, gpu_mstep

pytestmark = pytest.mark.gpu

ROWS = 20_000


def _slices():
    w = g.WORKLOADS["large"]
    mix = g.Mixture(w)
    starts = [0, w.n // 2, w.n - ROWS]
    xs = [mix.rows(s, s + ROWS) for s in starts]
    init = g.init_rows(w)
    means = np.concatenate([mix.rows(int(r), int(r) + 1) for r in init]).astype(np.float32)
    allx = np.concatenate(xs).astype(np.float64)
    var = np.tile(allx.var(axis=0), (w.k, 1)).astype(np.float32)
    wt = np.full(w.k, 1.0 / w.k, dtype=np.float32)
    return starts, xs, (wt, means, var)


def test_large_workload_slices_teacher_forced():
    starts, xs, th = _slices()
    sts = []
    for s, x in zip(starts, xs):
        ref = oracle.iterate(x, *th)
        st = gpu_estep(x, *th)
        r1 = check_stats(st, ref, f"rows {s}..")
        w2, mu2, var2 = gpu_mstep(st, float(x.shape[0]), *th)
        r2 = check_params(w2, mu2, var2, ref, x.shape[0], f"rows {s}..")
        print(f"  rows {s}+{ROWS}: {r1} {r2}", flush=True)
        sts.append(st)
    whole = gpu_estep(np.concatenate(xs), *th)
    # the dense part of the statistics is summed in fp32 runs whose boundaries depend on the
    # row count, so slices and their union agree to fp32 rounding of that part
    for key in ("nk", "s", "q"):
        tot = sum(st[key] for st in sts)
        np.testing.assert_allclose(tot, whole[key], rtol=1e-6, atol=1e-6)
    assert sum(st["loglik"] for st in sts) == pytest.approx(whole["loglik"], rel=1e-9)
