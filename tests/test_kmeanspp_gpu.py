"""GPU k-means++ seeding against the checker: with the same uniforms the chosen rows must be
identical draw by draw while a draw is decisive.

The checker sums D^2 plainly (over the dimensions in order, the running sum over the rows in
order); the GPU uses its own fixed order (strided partial sums, blocks of runs).  The two
running sums differ by rounding alone: each D^2 by at most about (d + 4) u relative, a sum of
n non-negative terms by at most n u of the total (u = 2^-53), so the running sums of the two
sides differ by less than BOUND = 4 (n + d) 2^-53 of the total.  Draw t is decisive when the
checker's margin (how far u_t * total lies inside the picked row's interval, relative to the
total) exceeds BOUND; there the picks must be equal.  Later draws depend on earlier ones, so the
comparison stops at the first draw that is not decisive; the tests require that none is hit
(random uniforms land within 1e-10 of a boundary with probability about 1e-10 n)."""
import sys

import numpy as np
import pytest

import gmm_synth as g
import oracle

pytestmark = pytest.mark.gpu


def _check_picks(got, ridx, margin, n, d, label):
    bound = 4.0 * (n + d) * 2.0 ** -53
    k = len(ridx)
    checked = 0
    for t in range(k):
        if not margin[t] > bound:
            break
        assert got[t] == ridx[t], f"{label}: draw {t} picked {got[t]}, checker {ridx[t]} " \
                                  f"(margin {margin[t]:.3e})"
        checked += 1
    print(f"  {label}: {checked} of {k} draws decisive and equal (bound {bound:.2e})", flush=True)
    assert checked == k, f"{label}: draw {checked} not decisive (margin {margin[checked]:.3e})"


@pytest.mark.parametrize("n,d,kt,k,seed", [(5000, 16, 8, 50, 1), (100003, 128, 64, 64, 2),
                                           (9000, 300, 12, 40, 3), (3 * 4096, 7, 5, 100, 4),
                                           (700, 1024, 3, 20, 5)])
def test_kmeanspp_matches_checker(n, d, kt, k, seed):
    import torch
    import paper_2606_10896_amd as gmm
    w = g.custom(f"kpp{n}_{d}", n, d, kt, kt, data_seed=seed, init_seed=seed)
    x, _ = g.make(w)
    u = np.random.default_rng(100 + seed).random(k)
    print(f"  k-means++ n={n} d={d} k={k}", flush=True)
    sys.stdout.flush()
    ridx, rcen, mg = oracle.kmeanspp(x, k, u, want_margin=True)
    xd = torch.from_numpy(x).cuda()
    ud = torch.from_numpy(u).cuda()
    idx = torch.full((k,), -1, dtype=torch.int64, device="cuda")
    cen = torch.zeros(k, d, dtype=torch.float32, device="cuda")
    gmm.gmm_kmeanspp(xd, ud, idx, cen)
    torch.cuda.synchronize()
    got = idx.cpu().numpy()
    _check_picks(got, ridx, mg, n, d, f"n={n} d={d} k={k}")
    np.testing.assert_array_equal(cen.cpu().numpy(), x[got])


def test_kmeanspp_duplicate_rows():
    import torch
    import paper_2606_10896_amd as gmm
    rng = np.random.default_rng(9)
    base = rng.standard_normal((6, 12)).astype(np.float32)
    x = np.repeat(base, 1500, axis=0)          # 9000 rows, 6 distinct
    u = rng.random(8)
    ridx, _, mg = oracle.kmeanspp(x, 8, u, want_margin=True)
    idx = torch.full((8,), -1, dtype=torch.int64, device="cuda")
    cen = torch.zeros(8, 12, dtype=torch.float32, device="cuda")
    gmm.gmm_kmeanspp(torch.from_numpy(x).cuda(), torch.from_numpy(u).cuda(), idx, cen)
    torch.cuda.synchronize()
    got = idx.cpu().numpy()
    _check_picks(got, ridx, mg, x.shape[0], 12, "duplicate rows")
    assert len(set((got[:6] // 1500).tolist())) == 6   # the first six cover the distinct rows
