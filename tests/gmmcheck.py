"""Helpers shared by the GPU tests: device wrappers around the C ABI and the
parity tolerances.

Tolerances (fp32 path, against the fp64 checker, same fp32 parameters into
both):
  N_k      |gpu - ref| <= 1e-4 * max(N_k, 1)
  mu_kd    |gpu - ref| <= 1e-4 * max(|mu_kd|, sigma_kd)     where ref N_k >= 1
  var_kd   |gpu - ref| <= 1e-4 * var_kd                      where ref N_k >= 1
  LL       |gpu - ref| <= 1e-5 * |LL|
Components with N_k < 1 are excluded from the mean and variance checks: their
statistics are dominated by responsibilities below fp32's range.
"""
from __future__ import annotations

import numpy as np

TOL_N = 1e-4
TOL_MU = 1e-4
TOL_VAR = 1e-4
TOL_LL = 1e-5


def to_dev(*arrays, device="cuda"):
    import torch
    return [torch.from_numpy(np.ascontiguousarray(a)).to(device) for a in arrays]


def gpu_estep(x, w, mu, var, xd=None, ws=None):
    """GPU statistics at fp32 parameters (numpy in, numpy fp64 out)."""
    import torch
    import paper_2606_10896_amd as gmm
    if xd is None:
        (xd,) = to_dev(x)
    n, d = xd.shape
    k = w.shape[0]
    wd, mud, vd = to_dev(w, mu, var)
    nk = torch.zeros(k, dtype=torch.float64, device="cuda")
    s = torch.zeros(k, d, dtype=torch.float64, device="cuda")
    q = torch.zeros(k, d, dtype=torch.float64, device="cuda")
    ll = torch.zeros(1, dtype=torch.float64, device="cuda")
    if ws is None:
        ws = gmm.workspace(n, d, k)
    gmm.gmm_estep_accumulate(xd, wd, mud, vd, nk, s, q, ll, ws)
    torch.cuda.synchronize()
    return dict(nk=nk.cpu().numpy(), s=s.cpu().numpy(), q=q.cpu().numpy(), loglik=ll.item())


def gpu_mstep(st, n_total, w, mu, var, var_floor=1e-6):
    import torch
    import paper_2606_10896_amd as gmm
    nk, s, q = to_dev(st["nk"], st["s"], st["q"])
    wd, mud, vd = to_dev(w, mu, var)
    gmm.gmm_mstep(nk, s, q, n_total, wd, mud, vd, var_floor=var_floor)
    torch.cuda.synchronize()
    return wd.cpu().numpy(), mud.cpu().numpy(), vd.cpu().numpy()


def gpu_fit(x, w, mu, var, n_iters, var_floor=1e-6, xd=None, ws=None):
    import torch
    import paper_2606_10896_amd as gmm
    if xd is None:
        (xd,) = to_dev(x)
    n, d = xd.shape
    k = w.shape[0]
    wd, mud, vd = to_dev(w, mu, var)
    hist = torch.zeros(max(n_iters, 1), dtype=torch.float64, device="cuda")
    if ws is None:
        ws = gmm.workspace(n, d, k)
    gmm.gmm_fit(xd, wd, mud, vd, n_iters, hist, ws, var_floor=var_floor)
    torch.cuda.synchronize()
    return wd.cpu().numpy(), mud.cpu().numpy(), vd.cpu().numpy(), hist.cpu().numpy()[:n_iters]


def check_stats(gpu, ref, label=""):
    """N_k and LL against the checker; returns a short report string."""
    nk_ref = ref["nk"]
    err_n = np.abs(gpu["nk"] - nk_ref) / np.maximum(nk_ref, 1.0)
    assert err_n.max() <= TOL_N, f"{label} N_k: max rel err {err_n.max():.3e} at {err_n.argmax()}"
    err_ll = abs(gpu["loglik"] - ref["loglik"]) / abs(ref["loglik"])
    assert err_ll <= TOL_LL, f"{label} LL: rel err {err_ll:.3e} ({gpu['loglik']} vs {ref['loglik']})"
    return f"N {err_n.max():.2e} LL {err_ll:.2e}"


def check_params(w, mu, var, ref, n_total, label=""):
    """M-step results against the checker's Theta_{t+1} (fp64).  Weights are N_k / N, so they
    carry the N_k tolerance (plus fp32 storage rounding)."""
    nk_ref = ref["nk"]
    live = nk_ref >= 1.0
    rw = ref["weights"]
    err_w = np.abs(w - rw) / np.maximum(rw, 1.0 / n_total)
    assert err_w.max() <= TOL_N + 1e-7, f"{label} weights: {err_w.max():.3e}"
    sig = np.sqrt(ref["vars"])
    err_mu = np.abs(mu - ref["means"]) / np.maximum(np.abs(ref["means"]), sig)
    err_mu = np.where(live[:, None], err_mu, 0.0)
    i = np.unravel_index(err_mu.argmax(), err_mu.shape)
    assert err_mu.max() <= TOL_MU, f"{label} means: {err_mu.max():.3e} at {i}"
    err_v = np.abs(var - ref["vars"]) / ref["vars"]
    err_v = np.where(live[:, None], err_v, 0.0)
    i = np.unravel_index(err_v.argmax(), err_v.shape)
    assert err_v.max() <= TOL_VAR, (f"{label} vars: {err_v.max():.3e} at {i} "
                                    f"(gpu {var[i]}, ref {ref['vars'][i]}, Nk {nk_ref[i[0]]})")
    return f"mu {err_mu.max():.2e} var {err_v.max():.2e}"
