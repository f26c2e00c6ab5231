"""The N = 1e8, D = 128, K = 1024 workload (51.2 GB of points resident in HBM, the paper's
Table 1 row N = 100M; its Limitations section notes the kernel validated at 1e8): one
gmm_estep_accumulate over all 1e8 rows against the sum of calls over 4,194,304-row views of the
same tensor, at the random-point initialisation and after two EM iterations.

Row offsets reach N * D = 1.28e10 > 2^31 in the whole-set call only, and its statistics chunks
hold 781,250 points (30,000 in the views), so the two sides share no launch shape; the checker
itself is run on row slices of this workload by test_large_slices_gpu.py.  The two sides differ
by the rounding of the dense statistics pass alone (where its fp32 runs split, and the order of
the fp64 partial sums), a few 1e-7 of N_k here; the bound used is 2e-5, five times tighter than
the parity tolerance against the checker, while a wrong row offset moves whole points."""
import sys
import time

import numpy as np
import pytest

import gmm_synth as g

pytestmark = pytest.mark.gpu

VIEW = 1 << 22
TOL = 2e-5


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def large():
    import torch
    import bench
    t0 = time.time()
    w = g.WORKLOADS["large"]
    dev = torch.device("cuda:0")
    x, mix, colsum, colsq = bench.load_data(w, dev)
    th0 = g.random_point_init(w, mix, colsum, colsq)
    _say(f"  large workload resident ({time.time() - t0:.1f}s)")
    yield w, x, th0
    del x
    torch.cuda.empty_cache()


def _stats(x, th, rows, ws):
    """Statistics of x at th from gmm_estep_accumulate calls over views of `rows` rows."""
    import torch
    import paper_2606_10896_amd as gmm
    n, d = x.shape
    k = th[0].shape[0]
    dev = x.device
    wt, mu, var = (torch.from_numpy(np.ascontiguousarray(a)).to(dev) for a in th)
    nk = torch.zeros(k, dtype=torch.float64, device=dev)
    s = torch.zeros(k, d, dtype=torch.float64, device=dev)
    q = torch.zeros(k, d, dtype=torch.float64, device=dev)
    ll = torch.zeros(1, dtype=torch.float64, device=dev)
    for r0 in range(0, n, rows):
        gmm.gmm_estep_accumulate(x[r0:r0 + rows], wt, mu, var, nk, s, q, ll, ws)
    torch.cuda.synchronize()
    return nk.cpu().numpy(), s.cpu().numpy(), q.cpu().numpy(), ll.item()


@pytest.mark.timeout(1100)
def test_large_workload_whole_equals_sum_of_views(large):
    import torch
    import paper_2606_10896_amd as gmm
    t0 = time.time()
    w, x, th0 = large
    dev = x.device
    n, d, k = w.n, w.d, w.k
    ws_all = gmm.workspace(n, d, k, device=dev)
    ws_view = gmm.workspace(VIEW, d, k, device=dev)

    def stats(th, views):
        return _stats(x, th, VIEW, ws_view) if views else _stats(x, th, n, ws_all)

    # Theta_2: two EM iterations of the library from Theta_0
    wt, mu, var = (torch.from_numpy(a).to(dev) for a in th0)
    hist = torch.zeros(2, dtype=torch.float64, device=dev)
    gmm.gmm_fit(x, wt, mu, var, 2, hist, ws_all)
    torch.cuda.synchronize()
    th2 = (wt.cpu().numpy(), mu.cpu().numpy(), var.cpu().numpy())
    for label, th in (("theta0", th0), ("theta2", th2)):
        a_nk, a_s, a_q, a_ll = stats(th, views=False)
        b_nk, b_s, b_q, b_ll = stats(th, views=True)
        assert abs(a_nk.sum() - n) <= 1e-6 * n
        e_n = np.abs(a_nk - b_nk) / np.maximum(a_nk, 1.0)
        # S_kd against its natural scale sqrt(N_k Q_kd) >= sum_i r_ik |x_id| (Cauchy-Schwarz)
        e_s = np.abs(a_s - b_s) / np.maximum(np.sqrt(np.maximum(a_nk, 1.0)[:, None] * a_q), 1e-30)
        e_q = np.abs(a_q - b_q) / np.maximum(a_q, 1e-30)
        e_ll = abs(a_ll - b_ll) / abs(a_ll)
        _say(f"  {label}: whole vs views: N_k {e_n.max():.2e}  S {e_s.max():.2e}  "
             f"Q {e_q.max():.2e}  LL {e_ll:.2e}  ({time.time() - t0:.1f}s)")
        assert e_n.max() <= TOL and e_s.max() <= TOL and e_q.max() <= TOL
        assert e_ll <= 1e-9


@pytest.mark.timeout(1100)
def test_large_workload_from_pageable_memory_through_the_ring(large):
    """X of the 1e8-row workload in ordinary host memory (51.2 GB, more than could be pinned
    whole), streamed through a ring of three page-locked 4,194,304-row slots by
    gmm_estep_accumulate_ring: bit for bit the statistics of gmm_estep_accumulate over the
    resident 4,194,304-row views."""
    import torch
    import paper_2606_10896_amd as gmm
    w, x, th0 = large
    dev = x.device
    n, d, k = w.n, w.d, w.k
    t0 = time.time()
    xh = np.empty((n, d), dtype=np.float32)
    for r0 in range(0, n, VIEW):
        xh[r0:r0 + VIEW] = x[r0:r0 + VIEW].cpu().numpy()
    _say(f"  pageable host copy of X ({time.time() - t0:.1f}s)")
    ws = gmm.workspace(VIEW, d, k, device=dev)
    ref = _stats(x, th0, VIEW, ws)
    ring = torch.empty((3, VIEW, d), dtype=torch.float32, pin_memory=True)
    staging = torch.empty(2 * VIEW * d, dtype=torch.float32, device=dev)
    copy = torch.cuda.Stream()
    wt, mu, var = (torch.from_numpy(np.ascontiguousarray(a)).to(dev) for a in th0)
    for rep in range(2):
        nk = torch.zeros(k, dtype=torch.float64, device=dev)
        s = torch.zeros(k, d, dtype=torch.float64, device=dev)
        q = torch.zeros(k, d, dtype=torch.float64, device=dev)
        ll = torch.zeros(1, dtype=torch.float64, device=dev)
        torch.cuda.synchronize()
        t1 = time.time()
        gmm.gmm_estep_accumulate_ring(xh, n, wt, mu, var, nk, s, q, ll, VIEW, ring, staging, ws,
                                      copy_stream=copy)
        torch.cuda.synchronize()
        dt = time.time() - t1
        _say(f"  ring E-step from pageable memory: {dt * 1e3:.0f} ms, "
             f"{4.0 * n * d / dt / 1e9:.1f} GB/s of X")
        got = (nk.cpu().numpy(), s.cpu().numpy(), q.cpu().numpy(), ll.item())
        for a, b, name in zip(got, ref, ("N_k", "S", "Q", "LL")):
            assert np.array_equal(a, b), f"pass {rep}: {name} differs from the resident views"
