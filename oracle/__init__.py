"""CPU checker (fp64) for the diagonal-GMM EM iteration — TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The GPU library never calls, links or
loads it, and it shares no code with the GPU path.

The arithmetic lives in ``oracle.c`` (plain fp64 loops; see its header for
the definitions and the paper passages they follow).  ``brute.py`` holds a
pure-Python enumeration used to pin it on tiny inputs.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_lib = None

#: variance floor used when none is given (absolute, applied after the M-step)
DEFAULT_VAR_FLOOR = 1e-6


def build_lib(force: bool = True) -> str:
    """Compile ``oracle.c`` into ``liboracle.so`` (gcc -O2, plain C)."""
    src = os.path.join(_HERE, "oracle.c")
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + ".tmp"
        subprocess.check_call(["gcc", "-O2", "-std=gnu11", "-fPIC", "-shared", "-o", tmp, src,
                               "-lm", "-lpthread"])
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build_lib(force=False)
        lib = ctypes.CDLL(_LIB_PATH)
        vp, i64, i32, f64 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_double
        lib.oracle_estep.argtypes = [vp, i64, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp, i32]
        lib.oracle_estep.restype = None
        lib.oracle_iterate.argtypes = [vp, i64, i32, i32, vp, vp, vp, f64, vp, vp, vp, vp, vp, vp,
                                       vp, i32]
        lib.oracle_iterate.restype = None
        lib.oracle_logdens.argtypes = [vp, i64, i32, i32, vp, vp, vp, vp, vp]
        lib.oracle_logdens.restype = None
        lib.oracle_assign_topk.argtypes = [vp, i64, i32, i32, vp, vp, vp, i32, f64, vp, vp, i32,
                                           vp, vp, i32]
        lib.oracle_assign_topk.restype = ctypes.c_int
        lib.oracle_kmeans.argtypes = [vp, i64, i32, i32, i32, f64, vp, vp, vp, vp, vp, vp, vp]
        lib.oracle_kmeans.restype = None
        lib.oracle_kmeanspp.argtypes = [vp, i64, i32, i32, vp, vp, vp, vp]
        lib.oracle_kmeanspp.restype = None
        lib.oracle_iso_estep.argtypes = [vp, i64, i32, i32, vp, vp, vp, vp, vp, vp, vp, i32]
        lib.oracle_iso_estep.restype = None
        lib.oracle_iso_iterate.argtypes = [vp, i64, i32, i32, vp, vp, vp, f64, vp, vp, vp, vp,
                                           vp, vp, vp, i32]
        lib.oracle_iso_iterate.restype = None
        _lib = lib
    return _lib


def _p(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _f32(a):
    return np.ascontiguousarray(a, dtype=np.float32)


def default_threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def _theta(weights, means, variances):
    w, mu, var = _f32(weights), _f32(means), _f32(variances)
    k, d = mu.shape
    assert w.shape == (k,) and var.shape == (k, d)
    return w, mu, var, k, d


def estep(x, weights, means, variances, nthreads=None, want_logz=False):
    """E-step statistics at the given fp32 parameters, fp64 results.

    Returns dict(nk[K], s[K,D], q[K,D], loglik, [logz[N]])."""
    x = _f32(x)
    w, mu, var, k, d = _theta(weights, means, variances)
    n = x.shape[0]
    assert x.shape == (n, d)
    nk = np.zeros(k)
    s = np.zeros((k, d))
    q = np.zeros((k, d))
    ll = np.zeros(1)
    logz = np.zeros(n) if want_logz else None
    _load().oracle_estep(_p(x), n, d, k, _p(w), _p(mu), _p(var), _p(nk), _p(s), _p(q), _p(ll),
                         _p(logz), nthreads or default_threads())
    out = dict(nk=nk, s=s, q=q, loglik=float(ll[0]))
    if want_logz:
        out["logz"] = logz
    return out


def iterate(x, weights, means, variances, var_floor=DEFAULT_VAR_FLOOR, nthreads=None):
    """One EM iteration at Theta_t.  Returns dict(weights, means, vars (fp64, Theta_{t+1}),
    loglik (= LL(Theta_t)), nk, s, q)."""
    x = _f32(x)
    w, mu, var, k, d = _theta(weights, means, variances)
    n = x.shape[0]
    assert x.shape == (n, d)
    w1, mu1, var1 = np.zeros(k), np.zeros((k, d)), np.zeros((k, d))
    nk, s, q, ll = np.zeros(k), np.zeros((k, d)), np.zeros((k, d)), np.zeros(1)
    _load().oracle_iterate(_p(x), n, d, k, _p(w), _p(mu), _p(var), float(var_floor), _p(w1),
                           _p(mu1), _p(var1), _p(nk), _p(s), _p(q), _p(ll),
                           nthreads or default_threads())
    return dict(weights=w1, means=mu1, vars=var1, loglik=float(ll[0]), nk=nk, s=s, q=q)


def fit(x, weights, means, variances, n_iters, var_floor=DEFAULT_VAR_FLOOR, nthreads=None,
        keep_thetas=False):
    """n_iters EM iterations from Theta_0.  Parameters are rounded to fp32 between iterations,
    as the GPU library stores them.  Returns dict(weights, means, vars (fp32, Theta_T),
    loglik_hist[n_iters] (LL(Theta_t)), thetas (list of fp32 Theta_t, t < T) if keep_thetas)."""
    th = (_f32(weights), _f32(means), _f32(variances))
    hist = np.zeros(n_iters)
    thetas = []
    for t in range(n_iters):
        if keep_thetas:
            thetas.append(th)
        r = iterate(x, *th, var_floor=var_floor, nthreads=nthreads)
        hist[t] = r["loglik"]
        th = (_f32(r["weights"]), _f32(r["means"]), _f32(r["vars"]))
    out = dict(weights=th[0], means=th[1], vars=th[2], loglik_hist=hist)
    if keep_thetas:
        out["thetas"] = thetas
    return out


def logdens(x, weights, means, variances):
    """Direct-form log-densities l[N,K] (log pi_k included) and log Z[N], fp64."""
    x = _f32(x)
    w, mu, var, k, d = _theta(weights, means, variances)
    n = x.shape[0]
    l = np.zeros((n, k))
    lz = np.zeros(n)
    _load().oracle_logdens(_p(x), n, d, k, _p(w), _p(mu), _p(var), _p(l), _p(lz))
    return l, lz


def assign_topk(x, weights, means, variances, m, tau, mr=0, nthreads=None):
    """Top-m multi-assignment.  Returns (idx int32 [N,m], resp fp32 [N,m]) and, if mr > 0,
    also (ridx [N,mr], rresp fp64 [N,mr]): the top-mr components with no tau rule."""
    x = _f32(x)
    w, mu, var, k, d = _theta(weights, means, variances)
    n = x.shape[0]
    idx = np.zeros((n, m), dtype=np.int32)
    resp = np.zeros((n, m), dtype=np.float32)
    ridx = np.zeros((n, mr), dtype=np.int32) if mr else None
    rresp = np.zeros((n, mr)) if mr else None
    rc = _load().oracle_assign_topk(_p(x), n, d, k, _p(w), _p(mu), _p(var), int(m), float(tau),
                                    _p(idx), _p(resp), int(mr), _p(ridx), _p(rresp),
                                    nthreads or default_threads())
    if rc != 0:
        raise ValueError("bad m / mr")
    if mr:
        return idx, resp, ridx, rresp
    return idx, resp


# ---------------------------------------------------------------- isotropic model (Sec. 2)
def _theta_iso(weights, means, variances):
    w, mu, var = _f32(weights), _f32(means), _f32(variances)
    k, d = mu.shape
    assert w.shape == (k,) and var.shape == (k,)
    return w, mu, var, k, d


def iso_estep(x, weights, means, variances, nthreads=None):
    """Isotropic E-step statistics (one scalar variance per component), fp64:
    dict(nk[K], s[K,D], q[K] = sum r ||x||^2, loglik)."""
    x = _f32(x)
    w, mu, var, k, d = _theta_iso(weights, means, variances)
    n = x.shape[0]
    assert x.shape == (n, d)
    nk, s, q, ll = np.zeros(k), np.zeros((k, d)), np.zeros(k), np.zeros(1)
    _load().oracle_iso_estep(_p(x), n, d, k, _p(w), _p(mu), _p(var), _p(nk), _p(s), _p(q),
                             _p(ll), nthreads or default_threads())
    return dict(nk=nk, s=s, q=q, loglik=float(ll[0]))


def iso_iterate(x, weights, means, variances, var_floor=DEFAULT_VAR_FLOOR, nthreads=None):
    """One isotropic EM iteration.  Returns dict(weights, means, vars[K] (fp64, Theta_{t+1}),
    loglik (= LL(Theta_t)), nk, s, q[K])."""
    x = _f32(x)
    w, mu, var, k, d = _theta_iso(weights, means, variances)
    n = x.shape[0]
    assert x.shape == (n, d)
    w1, mu1, var1 = np.zeros(k), np.zeros((k, d)), np.zeros(k)
    nk, s, q, ll = np.zeros(k), np.zeros((k, d)), np.zeros(k), np.zeros(1)
    _load().oracle_iso_iterate(_p(x), n, d, k, _p(w), _p(mu), _p(var), float(var_floor), _p(w1),
                               _p(mu1), _p(var1), _p(nk), _p(s), _p(q), _p(ll),
                               nthreads or default_threads())
    return dict(weights=w1, means=mu1, vars=var1, loglik=float(ll[0]), nk=nk, s=s, q=q)


def iso_fit(x, weights, means, variances, n_iters, var_floor=DEFAULT_VAR_FLOOR, nthreads=None,
            keep_thetas=False):
    """n_iters isotropic EM iterations from Theta_0 (fp32 parameters between iterations)."""
    th = (_f32(weights), _f32(means), _f32(variances))
    hist = np.zeros(n_iters)
    thetas = []
    for t in range(n_iters):
        if keep_thetas:
            thetas.append(th)
        r = iso_iterate(x, *th, var_floor=var_floor, nthreads=nthreads)
        hist[t] = r["loglik"]
        th = (_f32(r["weights"]), _f32(r["means"]), _f32(r["vars"]))
    out = dict(weights=th[0], means=th[1], vars=th[2], loglik_hist=hist)
    if keep_thetas:
        out["thetas"] = thetas
    return out


# ---------------------------------------------------------------- k-means++ seeding
def kmeanspp(x, k, u, want_margin=False):
    """k-means++ seeding with the given uniforms u[k] in [0, 1): D^2 sampling by inversion
    against the running sum in row order (see oracle.c).  Returns (rows int64 [k], centres
    fp32 [k, d]) and, with want_margin, also margin fp64 [k]: how far each draw's target lies
    inside the picked row's interval of the running sum, relative to the total (+inf for the
    first centre and a zero total)."""
    x = _f32(x)
    n, d = x.shape
    u = np.ascontiguousarray(u, dtype=np.float64)
    assert u.shape == (k,) and np.all((u >= 0.0) & (u < 1.0))
    idx = np.zeros(k, dtype=np.int64)
    cen = np.zeros((k, d), dtype=np.float32)
    mg = np.zeros(k)
    _load().oracle_kmeanspp(_p(x), n, d, k, _p(u), _p(idx), _p(cen), _p(mg))
    if want_margin:
        return idx, cen, mg
    return idx, cen


def kmeans(x, centres, variances, n_iters, var_floor=DEFAULT_VAR_FLOOR):
    """k-means warm start: n_iters Lloyd iterations from `centres` (centres rounded to fp32
    after every move, as the GPU stores them), then the hard-assignment mixture (see oracle.c).
    Returns dict(centres (fp64, after n_iters moves), weights, means, vars (fp64), assign)."""
    x = _f32(x)
    n, d = x.shape
    c0 = _f32(centres)
    k = c0.shape[0]
    var = _f32(variances)
    assert c0.shape == (k, d) and var.shape == (k, d)
    cen, w1, mu1, var1 = np.zeros((k, d)), np.zeros(k), np.zeros((k, d)), np.zeros((k, d))
    asg = np.zeros(n, dtype=np.int32)
    _load().oracle_kmeans(_p(x), n, d, k, int(n_iters), float(var_floor), _p(c0), _p(var),
                          _p(cen), _p(w1), _p(mu1), _p(var1), _p(asg))
    return dict(centres=cen, weights=w1, means=mu1, vars=var1, assign=asg)

