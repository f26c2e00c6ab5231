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

The reduced-precision calls (gmm_estep_accumulate_screened, gmm_fit_screened)
keep the screening pass's log-densities (split bf16 products) for every pair;
their tolerances, stated in the C header, are SCREENED_TOL:
  N_k 2e-3, mu_kd 2e-3 (same normalisations), LL 2e-5, and
  var_kd |gpu - ref| <= 5e-3 * (mu_kd^2 + var_kd)                 where ref N_k >= 1
A screened responsibility is within about e = 2^-21 (S + d) relative, S =
sum_j mu_j^2 / var_j of the components involved (S + d is 600 .. 1800 on the
tested inputs, e up to 9e-4).  The variance is Q/N - mu^2: a relative error
e of the weighted sums gives an error of about 3 e (mu^2 + var) in it, far
more than e var when a component narrows away from the origin.
"""
from __future__ import annotations

import numpy as np

TOL_N = 1e-4
TOL_MU = 1e-4
TOL_VAR = 1e-4
TOL_LL = 1e-5
EXACT_TOL = dict(n=TOL_N, mu=TOL_MU, var=TOL_VAR, ll=TOL_LL)
SCREENED_TOL = dict(n=2e-3, mu=2e-3, var=5e-3, ll=2e-5, var_second_moment=True)


def to_dev(*arrays, device="cuda"):
    import torch
    return [torch.from_numpy(np.ascontiguousarray(a)).to(device) for a in arrays]


def gpu_estep(x, w, mu, var, xd=None, ws=None, screened=False):
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
    fn = gmm.gmm_estep_accumulate_screened if screened else gmm.gmm_estep_accumulate
    fn(xd, wd, mud, vd, nk, s, q, ll, ws)
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


def gpu_fit(x, w, mu, var, n_iters, var_floor=1e-6, xd=None, ws=None, screened=False):
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
    fn = gmm.gmm_fit_screened if screened else gmm.gmm_fit
    fn(xd, wd, mud, vd, n_iters, hist, ws, var_floor=var_floor)
    torch.cuda.synchronize()
    return wd.cpu().numpy(), mud.cpu().numpy(), vd.cpu().numpy(), hist.cpu().numpy()[:n_iters]


def check_stats(gpu, ref, label="", tol=EXACT_TOL):
    """N_k and LL against the checker; returns a short report string."""
    nk_ref = ref["nk"]
    err_n = np.abs(gpu["nk"] - nk_ref) / np.maximum(nk_ref, 1.0)
    assert err_n.max() <= tol["n"], f"{label} N_k: max rel err {err_n.max():.3e} at {err_n.argmax()}"
    err_ll = abs(gpu["loglik"] - ref["loglik"]) / abs(ref["loglik"])
    assert err_ll <= tol["ll"], f"{label} LL: rel err {err_ll:.3e} ({gpu['loglik']} vs {ref['loglik']})"
    return f"N {err_n.max():.2e} LL {err_ll:.2e}"


def check_params(w, mu, var, ref, n_total, label="", tol=EXACT_TOL):
    """M-step results against the checker's Theta_{t+1} (fp64).  Weights are N_k / N, so they
    carry the N_k tolerance (plus fp32 storage rounding)."""
    nk_ref = ref["nk"]
    live = nk_ref >= 1.0
    rw = ref["weights"]
    err_w = np.abs(w - rw) / np.maximum(rw, 1.0 / n_total)
    assert err_w.max() <= tol["n"] + 1e-7, f"{label} weights: {err_w.max():.3e}"
    sig = np.sqrt(ref["vars"])
    err_mu = np.abs(mu - ref["means"]) / np.maximum(np.abs(ref["means"]), sig)
    err_mu = np.where(live[:, None], err_mu, 0.0)
    i = np.unravel_index(err_mu.argmax(), err_mu.shape)
    assert err_mu.max() <= tol["mu"], f"{label} means: {err_mu.max():.3e} at {i}"
    scale = ref["vars"] + ref["means"] ** 2 if tol.get("var_second_moment") else ref["vars"]
    err_v = np.abs(var - ref["vars"]) / scale
    err_v = np.where(live[:, None], err_v, 0.0)
    i = np.unravel_index(err_v.argmax(), err_v.shape)
    assert err_v.max() <= tol["var"], (f"{label} vars: {err_v.max():.3e} at {i} "
                                    f"(gpu {var[i]}, ref {ref['vars'][i]}, Nk {nk_ref[i[0]]})")
    return f"mu {err_mu.max():.2e} var {err_v.max():.2e}"


# ---- isotropic model (one variance per component)
def gpu_estep_iso(x, w, mu, var, xd=None, ws=None):
    import torch
    import paper_2606_10896_amd as gmm
    if xd is None:
        (xd,) = to_dev(x)
    n, d = xd.shape
    k = w.shape[0]
    wd, mud, vd = to_dev(w, mu, var)
    nk = torch.zeros(k, dtype=torch.float64, device="cuda")
    s = torch.zeros(k, d, dtype=torch.float64, device="cuda")
    q = torch.zeros(k, dtype=torch.float64, device="cuda")
    ll = torch.zeros(1, dtype=torch.float64, device="cuda")
    if ws is None:
        ws = gmm.workspace(n, d, k)
    gmm.gmm_estep_accumulate_iso(xd, wd, mud, vd, nk, s, q, ll, ws)
    torch.cuda.synchronize()
    return dict(nk=nk.cpu().numpy(), s=s.cpu().numpy(), q=q.cpu().numpy(), loglik=ll.item())


def gpu_mstep_iso(st, n_total, w, mu, var, var_floor=1e-6):
    import torch
    import paper_2606_10896_amd as gmm
    nk, s, q = to_dev(st["nk"], st["s"], st["q"])
    wd, mud, vd = to_dev(w, mu, var)
    gmm.gmm_mstep_iso(nk, s, q, n_total, wd, mud, vd, var_floor=var_floor)
    torch.cuda.synchronize()
    return wd.cpu().numpy(), mud.cpu().numpy(), vd.cpu().numpy()


def gpu_fit_iso(x, w, mu, var, n_iters, var_floor=1e-6, xd=None):
    import torch
    import paper_2606_10896_amd as gmm
    if xd is None:
        (xd,) = to_dev(x)
    n, d = xd.shape
    k = w.shape[0]
    wd, mud, vd = to_dev(w, mu, var)
    hist = torch.zeros(max(n_iters, 1), dtype=torch.float64, device="cuda")
    ws = gmm.workspace(n, d, k)
    gmm.gmm_fit_iso(xd, wd, mud, vd, n_iters, hist, ws, var_floor=var_floor)
    torch.cuda.synchronize()
    return wd.cpu().numpy(), mud.cpu().numpy(), vd.cpu().numpy(), hist.cpu().numpy()[:n_iters]


def check_params_iso(w, mu, var, ref, n_total, label=""):
    """Isotropic M-step against the checker: as check_params, with one variance per
    component (and sigma = sqrt(var_k) for every dimension of the mean)."""
    return check_params(w, mu, var[:, None], dict(ref, vars=ref["vars"][:, None]), n_total, label)


# ---- top-m assignment (Sec. 4.2 / 4.3)
MARGIN = 1e-6   # an index must match where the checker's top-m margin exceeds this
TOL_RESP = 1e-4


def gpu_assign(x, w, mu, var, m, tau, xd=None, ws=None):
    import torch
    import paper_2606_10896_amd as gmm
    if xd is None:
        (xd,) = to_dev(x)
    n, d = xd.shape
    k = w.shape[0]
    wd, mud, vd = to_dev(w, mu, var)
    idx = torch.full((n, m), -7, dtype=torch.int32, device="cuda")
    resp = torch.full((n, m), -7.0, dtype=torch.float32, device="cuda")
    if ws is None:
        ws = gmm.workspace(n, d, k, m)
    gmm.gmm_assign_topk(xd, wd, mud, vd, m, tau, idx, resp, ws)
    torch.cuda.synchronize()
    return idx.cpu().numpy(), resp.cpu().numpy()


def check_assign(gidx, gresp, ref, m, tau, label="", min_checked=0.9):
    """ref = oracle.assign_topk(..., mr=m+1).  Rank j of point i is checked where its margin
    min(r_(j-1) - r_(j), r_(j) - r_(j+1)) in the checker's fp64 responsibilities exceeds MARGIN
    (r_(0) = +inf) and, for j > 0, |r_(j) - tau| > MARGIN: there the index must be identical and
    the responsibility within TOL_RESP (an empty slot is -1 / 0 on both sides).  At least
    min_checked of the rank-1 entries must be decisive (later ranks often are not: two
    responsibilities below 1e-6 differ by less than the margin).  Returns the fraction of all
    (point, rank) pairs checked."""
    idx, resp, ridx, rresp = ref
    n = idx.shape[0]
    assert gidx.shape == (n, m) and gresp.shape == (n, m)
    rp = np.concatenate([np.full((n, 1), np.inf), rresp], axis=1)   # r_(0) = +inf
    checked = 0
    checked0 = 0
    bad = []
    for j in range(m):
        r = rp[:, j + 1]
        margin = np.minimum(rp[:, j] - r, r - rp[:, j + 2])
        ok = margin > MARGIN
        if j > 0:
            ok &= np.abs(r - tau) > MARGIN
        sel = np.nonzero(ok)[0]
        checked += sel.size
        if j == 0:
            checked0 = sel.size
        wrong = sel[gidx[sel, j] != idx[sel, j]]
        if wrong.size:
            i = wrong[0]
            bad.append(f"rank {j}: {wrong.size} index mismatches, e.g. point {i}: gpu "
                       f"{gidx[i]} ref {idx[i]} r {rresp[i]}")
        same = sel[gidx[sel, j] == idx[sel, j]]
        err = np.abs(gresp[same, j].astype(np.float64) - resp[same, j].astype(np.float64))
        if err.size and err.max() > TOL_RESP:
            i = same[err.argmax()]
            bad.append(f"rank {j}: resp err {err.max():.3e} at point {i}")
    assert not bad, f"{label}: " + "; ".join(bad)
    assert checked0 >= min_checked * n, \
        f"{label}: only {checked0 / n:.3f} of the rank-1 entries are decisive"
    return checked / (n * m)


# ---- depth of the dense statistics pass's fp32 runs
FOLD_POINTS = 4096   # queued points per fp32 run before the sums move into fp64


def queue_lower_bound(x, w, mu, var, chunk_rows, block=64, skip_top=8, window=50.0,
                      batch=20000):
    """A lower bound, per (64-component block, chunk of chunk_rows consecutive points), of the
    points the dense statistics pass queues for the block: the points holding a pair with
    r > 2^-window in the block that is not among the point's skip_top largest (the GPU stores
    its four largest exact pairs and leaves them out of the dense pass; every other pair above
    2^-64, up to the screening error of a few log2 units, marks its block).  Log-densities in
    fp64 by the expanded form with numpy (errors far below the 14 log2 units of slack between
    2^-50 and 2^-64).  Returns the largest count over (block, chunk)."""
    x = np.asarray(x, dtype=np.float64)
    n, d = x.shape
    k = mu.shape[0]
    iv = 1.0 / var.astype(np.float64)
    m64 = mu.astype(np.float64)
    with np.errstate(divide="ignore"):
        c = np.log(w.astype(np.float64)) - 0.5 * (np.log(2 * np.pi * var.astype(np.float64)).sum(1)
                                                  + (m64 * m64 * iv).sum(1))
    nb = (k + block - 1) // block
    nch = (n + chunk_rows - 1) // chunk_rows
    cnt = np.zeros((nb, nch), dtype=np.int64)
    for a in range(0, n, batch):
        xb = x[a:a + batch]
        l = c[None, :] + xb @ (m64 * iv).T - 0.5 * ((xb * xb) @ iv.T)
        mx = l.max(1, keepdims=True)
        lz = mx + np.log(np.exp(l - mx).sum(1, keepdims=True))
        lr2 = (l - lz) / np.log(2.0)
        top = np.argpartition(-lr2, skip_top, axis=1)[:, :skip_top]
        sig = lr2 > -window
        sig[np.arange(xb.shape[0])[:, None], top] = False
        pad = nb * block - k
        if pad:
            sig = np.concatenate([sig, np.zeros((sig.shape[0], pad), bool)], axis=1)
        marked = sig.reshape(sig.shape[0], nb, block).any(2)          # [rows, blocks]
        ch = (np.arange(a, a + xb.shape[0]) // chunk_rows)
        for j in np.unique(ch):
            cnt[:, j] += marked[ch == j].sum(0)
    return int(cnt.max())
