"""gmm_estep_accumulate_static (the E-step with the library's own static device workspace, for
callers that cannot allocate) against gmm_estep_accumulate on the same inputs, through the C
ABI: two calls in a row, the second with a smaller input, each compared with the parity
tolerances of the fp32 path (gmmcheck), and the second, whose workspace fits without shrinking
any split, bit for bit.  The static array keeps the first call's contents when the second
starts, so the second also shows that nothing is read before it is written."""
import ctypes
import sys

import numpy as np
import pytest

import gmm_synth as g
import oracle
from gmmcheck import check_stats, gpu_estep, to_dev

pytestmark = pytest.mark.gpu


def _static(x, w, mu, var):
    import torch
    import paper_2606_10896_amd as gmm
    lib = gmm.load_library()
    (xd,) = to_dev(x)
    wd, mud, vd = to_dev(w, mu, var)
    n, d = x.shape
    k = w.shape[0]
    nk = torch.zeros(k, dtype=torch.float64, device="cuda")
    s = torch.zeros(k, d, dtype=torch.float64, device="cuda")
    q = torch.zeros(k, d, dtype=torch.float64, device="cuda")
    ll = torch.zeros(1, dtype=torch.float64, device="cuda")
    p = lambda t: ctypes.c_void_p(t.data_ptr())
    rc = lib.gmm_estep_accumulate_static(p(xd), n, d, k, p(wd), p(mud), p(vd), p(nk), p(s),
                                         p(q), p(ll),
                                         ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert rc == gmm.GMM_OK, gmm.status_string(rc)
    torch.cuda.synchronize()
    return dict(nk=nk.cpu().numpy(), s=s.cpu().numpy(), q=q.cpu().numpy(), loglik=ll.item())


def test_static_estep_matches_the_workspace_call_twice():
    cases = [g.custom("st1", 300_000, 128, 256, 1024, data_seed=31, init_seed=3031),
             g.custom("st2", 7_000, 37, 12, 45, data_seed=32, init_seed=3032)]
    for i, spec in enumerate(cases):
        x, th = g.make(spec)
        print(f"  static call {i}: n={x.shape[0]} d={x.shape[1]} k={th[0].shape[0]}", flush=True)
        sys.stdout.flush()
        a = _static(x, *th)
        b = gpu_estep(x, *th)
        r = check_stats(a, b, f"static vs workspace call {i}")
        ds = np.abs(a["s"] - b["s"]).max() / np.abs(b["s"]).max()
        dq = np.abs(a["q"] - b["q"]).max() / np.abs(b["q"]).max()
        print(f"    {r}  S {ds:.2e}  Q {dq:.2e}", flush=True)
        assert ds <= 1e-4 and dq <= 1e-4
        if i == 1:
            for key in ("nk", "s", "q"):
                assert np.array_equal(a[key], b[key]), key
            assert a["loglik"] == b["loglik"]
            ref = oracle.estep(x, *th)
            print(f"    against the checker: {check_stats(a, ref, 'static vs checker')}",
                  flush=True)
