"""The IVF coarse-quantiser workload (N = 5e6 unit-normalised points, D = 768, K = 4096) on
row slices (start, middle and end of the data set, each generated on its own): teacher-forced
statistics against the fp64 checker at the random-point initialisation and after two checker
iterations, and top-2 multi-assignment with tau = 1/K.  The parameters use K rows of the
workload (its random-point initialisation rows) as means, uniform weights and the pooled
per-dimension population variance of the slices."""
import numpy as np
import pytest

import gmm_synth as g
import oracle
from gmmcheck import check_assign, check_params, check_stats, gpu_assign, gpu_estep, gpu_mstep

pytestmark = pytest.mark.gpu

ROWS = 2000


def _slices():
    w = g.WORKLOADS["ivf"]
    mix = g.Mixture(w)
    starts = [0, w.n // 2, w.n - ROWS]
    xs = [mix.rows(s, s + ROWS) for s in starts]
    init = g.init_rows(w)
    means = np.concatenate([mix.rows(int(r), int(r) + 1) for r in init]).astype(np.float32)
    allx = np.concatenate(xs).astype(np.float64)
    var = np.tile(allx.var(axis=0), (w.k, 1)).astype(np.float32)
    wt = np.full(w.k, 1.0 / w.k, dtype=np.float32)
    return w, starts, xs, (wt, means, var)


def test_ivf_slices_teacher_forced():
    w, starts, xs, th = _slices()
    for s, x in zip(starts, xs):
        thetas = [th]
        if s == starts[1]:
            f = oracle.fit(x, *th, 2, keep_thetas=True)
            thetas.append((f["weights"], f["means"], f["vars"]))
        for t, tht in enumerate(thetas):
            ref = oracle.iterate(x, *tht)
            st = gpu_estep(x, *tht)
            r1 = check_stats(st, ref, f"rows {s}.. t{t}")
            w2, mu2, var2 = gpu_mstep(st, float(x.shape[0]), *tht)
            r2 = check_params(w2, mu2, var2, ref, x.shape[0], f"rows {s}.. t{t}")
            print(f"  rows {s}+{ROWS} theta {t}: {r1} {r2}", flush=True)


def test_ivf_slice_assign_top2():
    w, starts, xs, th = _slices()
    x = xs[2]
    f = oracle.fit(x, *th, 2, keep_thetas=False)
    tht = (f["weights"], f["means"], f["vars"])
    ref = oracle.assign_topk(x, *tht, 2, w.tau, mr=3)
    gidx, gresp = gpu_assign(x, *tht, 2, w.tau)
    frac = check_assign(gidx, gresp, ref, 2, w.tau, "ivf slice top-2")
    print(f"  ivf assign: checked {frac:.4f} of ranks, kept per rank "
          f"{(gidx >= 0).sum(axis=0).tolist()}", flush=True)
