"""GPU k-means warm start against the checker: the same assignments wherever the nearest
centre is decisive (relative distance gap above 1e-6; these data have no closer ties), the
same centres after every move (fp32 storage of fp64 means), and the hard-assignment mixture
under the EM tolerances."""
import sys

import numpy as np
import pytest

import gmm_synth as g
import oracle
from gmmcheck import to_dev

pytestmark = pytest.mark.gpu


def _gap(x, centres):
    d2 = ((x.astype(np.float64)[:, None, :] - centres[None, :, :]) ** 2).sum(2)
    s = np.sort(d2, axis=1)
    return (s[:, 1] - s[:, 0]) / np.maximum(s[:, 0], 1e-30)


@pytest.mark.parametrize("n,d,kt,k,it", [(3000, 16, 8, 10, 5), (20000, 128, 30, 64, 4),
                                         (2500, 300, 6, 12, 3), (1200, 768, 5, 9, 2)])
def test_kmeans_matches_checker(n, d, kt, k, it):
    import torch
    import paper_2606_10896_amd as gmm
    w = g.custom(f"km{n}_{d}", n, d, kt, k, data_seed=31 + d, init_seed=41 + k)
    x, (w0, mu0, var0) = g.make(w)
    print(f"  k-means n={n} d={d} k={k} iterations={it}", flush=True)
    sys.stdout.flush()
    ref = oracle.kmeans(x, mu0, var0, it)
    xd, wd, mud, vd = to_dev(x, w0, mu0, var0)
    asg = torch.full((n,), -1, dtype=torch.int32, device="cuda")
    ws = gmm.workspace(n, d, k, 1)
    gmm.gmm_kmeans(xd, wd, mud, vd, it, asg, ws)
    torch.cuda.synchronize()
    a = asg.cpu().numpy()
    decisive = _gap(x, ref["centres"]) > 1e-6
    assert decisive.mean() > 0.99
    np.testing.assert_array_equal(a[decisive], ref["assign"][decisive])
    # the mixture from the last assignment
    live = ref["weights"] > 0
    np.testing.assert_allclose(wd.cpu().numpy(), ref["weights"], rtol=1e-6, atol=1e-7)
    mu = mud.cpu().numpy()
    sig = np.sqrt(ref["vars"])
    err_mu = np.abs(mu - ref["means"]) / np.maximum(np.abs(ref["means"]), sig)
    assert err_mu[live].max() <= 1e-5
    err_v = np.abs(vd.cpu().numpy() - ref["vars"]) / ref["vars"]
    assert err_v[live].max() <= 1e-4


def test_kmeans_zero_iterations_is_the_hard_mixture_of_the_given_centres():
    import torch
    import paper_2606_10896_amd as gmm
    w = g.custom("km0", 4000, 24, 6, 6, data_seed=3, init_seed=4)
    x, (w0, mu0, var0) = g.make(w)
    ref = oracle.kmeans(x, mu0, var0, 0)
    xd, wd, mud, vd = to_dev(x, w0, mu0, var0)
    asg = torch.full((4000,), -1, dtype=torch.int32, device="cuda")
    gmm.gmm_kmeans(xd, wd, mud, vd, 0, asg, gmm.workspace(4000, 24, 6, 1))
    torch.cuda.synchronize()
    np.testing.assert_array_equal(asg.cpu().numpy(), ref["assign"])
    np.testing.assert_allclose(wd.cpu().numpy(), ref["weights"], rtol=1e-6)
