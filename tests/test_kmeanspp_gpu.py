"""GPU k-means++ seeding against the checker: with the same uniforms every chosen row must be
identical (both sides fix the order of every sum, so each D^2 decision is the same)."""
import sys

import numpy as np
import pytest

import gmm_synth as g
import oracle

pytestmark = pytest.mark.gpu


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
    ridx, rcen = oracle.kmeanspp(x, k, u)
    xd = torch.from_numpy(x).cuda()
    ud = torch.from_numpy(u).cuda()
    idx = torch.full((k,), -1, dtype=torch.int64, device="cuda")
    cen = torch.zeros(k, d, dtype=torch.float32, device="cuda")
    gmm.gmm_kmeanspp(xd, ud, idx, cen)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(idx.cpu().numpy(), ridx)
    np.testing.assert_array_equal(cen.cpu().numpy(), rcen)


def test_kmeanspp_duplicate_rows():
    import torch
    import paper_2606_10896_amd as gmm
    rng = np.random.default_rng(9)
    base = rng.standard_normal((6, 12)).astype(np.float32)
    x = np.repeat(base, 1500, axis=0)          # 9000 rows, 6 distinct
    u = rng.random(8)
    ridx, _ = oracle.kmeanspp(x, 8, u)
    idx = torch.full((8,), -1, dtype=torch.int64, device="cuda")
    cen = torch.zeros(8, 12, dtype=torch.float32, device="cuda")
    gmm.gmm_kmeanspp(torch.from_numpy(x).cuda(), torch.from_numpy(u).cuda(), idx, cen)
    torch.cuda.synchronize()
    got = idx.cpu().numpy()
    np.testing.assert_array_equal(got, ridx)
    assert len(set((got[:6] // 1500).tolist())) == 6   # the first six cover the distinct rows
