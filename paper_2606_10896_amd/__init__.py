"""Python binding of ``libflashgmm.so``: the fused diagonal-GMM EM iteration on MI355X.

Argument marshalling only: every step of the computation runs in the HIP
kernels of ``csrc/flashgmm.hip``.  PyTorch provides the device memory (CUDA
tensors on ROCm) and the stream (``torch.cuda.current_stream()``); the entry
points take the same names and arguments as the C ABI in
``include/flashgmm.h``.  There is no CPU fallback: without the built library
every call raises.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libflashgmm.so")

GMM_OK = 0
GMM_ERR_INVALID_ARG = -1
GMM_ERR_UNSUPPORTED = -2
GMM_ERR_WORKSPACE = -3
GMM_ERR_DEVICE = -4
GMM_ERR_FILL = -5
GMM_MAX_D = 1024
GMM_MAX_K = 65535
GMM_MAX_M = 8

#: every symbol the C ABI exports
EXPORTS = ("gmm_status_string", "gmm_workspace_bytes", "gmm_estep_accumulate", "gmm_mstep",
           "gmm_fit", "gmm_assign_topk", "gmm_kmeanspp_workspace_bytes", "gmm_kmeanspp",
           "gmm_kmeans",
           "gmm_estep_accumulate_streamed",
           "gmm_estep_accumulate_iso", "gmm_mstep_iso", "gmm_fit_iso", "gmm_timing_enable",
           "gmm_timing_read", "gmm_estep_accumulate_screened", "gmm_fit_screened",
           "gmm_set_stats_chunk_limit", "gmm_estep_accumulate_static",
           "gmm_estep_accumulate_ring", "gmm_fill_pageable")

_lib = None


class GMMError(RuntimeError):
    def __init__(self, fn: str, status: int):
        self.status = status
        super().__init__(f"{fn} failed: {status_string(status)} ({status})")


def load_library():
    """Loads libflashgmm.so; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with paper_2606_10896_amd.build "
                           "(no CPU fallback exists)")
    # torch first: the library must bind to the HIP runtime that allocates the tensors it
    # is given (loading it first would pull in a second runtime, whose device pointers
    # differ from torch's)
    import torch  # noqa: F401
    lib = ctypes.CDLL(LIB_PATH)
    vp, i64, i32, f32, f64 = (ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_float,
                              ctypes.c_double)
    lib.gmm_status_string.argtypes = [ctypes.c_int]
    lib.gmm_status_string.restype = ctypes.c_char_p
    lib.gmm_workspace_bytes.argtypes = [i64, i32, i32, i32]
    lib.gmm_workspace_bytes.restype = ctypes.c_size_t
    lib.gmm_estep_accumulate.argtypes = [vp, i64, i32, i32, vp, vp, vp, vp, vp, vp, vp, vp,
                                         ctypes.c_size_t, vp]
    lib.gmm_estep_accumulate.restype = ctypes.c_int
    lib.gmm_mstep.argtypes = [vp, vp, vp, f64, i32, i32, f32, vp, vp, vp, vp]
    lib.gmm_mstep.restype = ctypes.c_int
    lib.gmm_fit.argtypes = [vp, i64, i32, i32, i32, f32, vp, vp, vp, vp, vp, ctypes.c_size_t, vp]
    lib.gmm_fit.restype = ctypes.c_int
    lib.gmm_estep_accumulate_screened.argtypes = lib.gmm_estep_accumulate.argtypes
    lib.gmm_estep_accumulate_screened.restype = ctypes.c_int
    lib.gmm_fit_screened.argtypes = lib.gmm_fit.argtypes
    lib.gmm_fit_screened.restype = ctypes.c_int
    lib.gmm_assign_topk.argtypes = [vp, i64, i32, i32, vp, vp, vp, i32, f32, vp, vp, vp,
                                    ctypes.c_size_t, vp]
    lib.gmm_assign_topk.restype = ctypes.c_int
    lib.gmm_kmeans.argtypes = [vp, i64, i32, i32, i32, f32, vp, vp, vp, vp, vp, ctypes.c_size_t,
                               vp]
    lib.gmm_kmeans.restype = ctypes.c_int
    lib.gmm_kmeanspp_workspace_bytes.argtypes = [i64]
    lib.gmm_kmeanspp_workspace_bytes.restype = ctypes.c_size_t
    lib.gmm_kmeanspp.argtypes = [vp, i64, i32, i32, vp, vp, vp, vp, ctypes.c_size_t, vp]
    lib.gmm_kmeanspp.restype = ctypes.c_int
    lib.gmm_estep_accumulate_streamed.argtypes = [vp, i64, i32, i32, vp, vp, vp, vp, vp, vp,
                                                  vp, i64, vp, vp, ctypes.c_size_t, vp, vp]
    lib.gmm_estep_accumulate_streamed.restype = ctypes.c_int
    lib.gmm_fill_pageable.argtypes = [vp, i64, i64, i32, vp]
    lib.gmm_fill_pageable.restype = ctypes.c_int
    lib.gmm_estep_accumulate_ring.argtypes = [vp, vp, i64, i32, i32, vp, vp, vp, vp, vp, vp, vp,
                                              i64, vp, i32, vp, vp, ctypes.c_size_t, vp, vp]
    lib.gmm_estep_accumulate_ring.restype = ctypes.c_int
    lib.gmm_estep_accumulate_iso.argtypes = lib.gmm_estep_accumulate.argtypes
    lib.gmm_estep_accumulate_iso.restype = ctypes.c_int
    lib.gmm_mstep_iso.argtypes = lib.gmm_mstep.argtypes
    lib.gmm_mstep_iso.restype = ctypes.c_int
    lib.gmm_fit_iso.argtypes = lib.gmm_fit.argtypes
    lib.gmm_fit_iso.restype = ctypes.c_int
    lib.gmm_timing_enable.argtypes = [ctypes.c_int]
    lib.gmm_timing_enable.restype = ctypes.c_int
    lib.gmm_timing_read.argtypes = [vp, i32, vp]
    lib.gmm_timing_read.restype = ctypes.c_int
    lib.gmm_estep_accumulate_static.argtypes = [vp, i64, i32, i32, vp, vp, vp, vp, vp, vp, vp,
                                                vp]
    lib.gmm_estep_accumulate_static.restype = ctypes.c_int
    lib.gmm_set_stats_chunk_limit.argtypes = [i32]
    lib.gmm_set_stats_chunk_limit.restype = ctypes.c_int
    _lib = lib
    return lib


def status_string(status: int) -> str:
    return load_library().gmm_status_string(int(status)).decode()


def workspace_bytes(n: int, d: int, k: int, m: int = 0) -> int:
    """Workspace size for (n, d, k); m > 0 sizes it for gmm_assign_topk."""
    return int(load_library().gmm_workspace_bytes(int(n), int(d), int(k), int(m)))


# ------------------------------------------------------------------ tensor helpers

def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _check(fn, rc):
    if rc != GMM_OK:
        raise GMMError(fn, rc)


def _dev(t, dtype, name, numel=None):
    """t as given, after checking that it is a contiguous CUDA tensor of `dtype` holding at
    least `numel` elements (the library reads and writes exactly the sizes (n, d, k) imply)."""
    import torch
    if not (isinstance(t, torch.Tensor) and t.is_cuda and t.dtype == dtype and t.is_contiguous()):
        raise TypeError(f"{name} must be a contiguous {dtype} CUDA tensor")
    if numel is not None and t.numel() < numel:
        raise ValueError(f"{name} holds {t.numel()} elements, {numel} needed")
    return t


def workspace(n: int, d: int, k: int, m: int = 0, device="cuda"):
    """A workspace tensor (uint8, 256-byte aligned by the caching allocator)."""
    import torch
    nb = workspace_bytes(n, d, k, m)
    if nb == 0:
        raise GMMError("gmm_workspace_bytes", GMM_ERR_UNSUPPORTED)
    return torch.empty(nb, dtype=torch.uint8, device=device)


def gmm_estep_accumulate(x, weights, means, variances, nk, s, q, loglik, ws, stream=None,
                         _fn="gmm_estep_accumulate"):
    """Adds the E-step statistics of x at (weights, means, variances) into fp64 nk, s, q and
    loglik (all CUDA tensors)."""
    import torch
    _dev(x, torch.float32, "x")
    n, d = x.shape
    k = weights.shape[0]
    rc = getattr(load_library(), _fn)(
        _ptr(x), n, d, k, _ptr(_dev(weights, torch.float32, "weights", k)),
        _ptr(_dev(means, torch.float32, "means", k * d)),
        _ptr(_dev(variances, torch.float32, "vars", k * d)),
        _ptr(_dev(nk, torch.float64, "nk", k)), _ptr(_dev(s, torch.float64, "s", k * d)),
        _ptr(_dev(q, torch.float64, "q", k * d)), _ptr(_dev(loglik, torch.float64, "loglik", 1)),
        _ptr(ws), ws.numel() if ws is not None else 0, _stream(stream))
    _check(_fn, rc)


def gmm_estep_accumulate_screened(x, weights, means, variances, nk, s, q, loglik, ws,
                                  stream=None):
    """gmm_estep_accumulate at the screening pass's precision (no fp64 refinement of the
    pairs that carry a point's mass); looser tolerances, stated in the C header."""
    gmm_estep_accumulate(x, weights, means, variances, nk, s, q, loglik, ws, stream,
                         _fn="gmm_estep_accumulate_screened")


def gmm_mstep(nk, s, q, n_total, weights, means, variances, var_floor=1e-6, stream=None):
    """M-step from fp64 statistics; updates fp32 weights/means/variances in place."""
    import torch
    k, d = means.shape
    rc = load_library().gmm_mstep(
        _ptr(_dev(nk, torch.float64, "nk", k)), _ptr(_dev(s, torch.float64, "s", k * d)),
        _ptr(_dev(q, torch.float64, "q", k * d)), float(n_total), d, k, float(var_floor),
        _ptr(_dev(weights, torch.float32, "weights", k)),
        _ptr(_dev(means, torch.float32, "means", k * d)),
        _ptr(_dev(variances, torch.float32, "vars", k * d)), _stream(stream))
    _check("gmm_mstep", rc)


def gmm_fit(x, weights, means, variances, n_iters, loglik_hist, ws, var_floor=1e-6, stream=None,
            _fn="gmm_fit"):
    """n_iters EM iterations; parameters updated in place, loglik_hist[t] = LL(Theta_t)."""
    import torch
    _dev(x, torch.float32, "x")
    n, d = x.shape
    k = weights.shape[0]
    rc = getattr(load_library(), _fn)(
        _ptr(x), n, d, k, int(n_iters), float(var_floor),
        _ptr(_dev(weights, torch.float32, "weights", k)),
        _ptr(_dev(means, torch.float32, "means", k * d)),
        _ptr(_dev(variances, torch.float32, "vars", k * d)),
        _ptr(_dev(loglik_hist, torch.float64, "loglik_hist", n_iters)), _ptr(ws),
        ws.numel() if ws is not None else 0, _stream(stream))
    _check(_fn, rc)


def gmm_fit_screened(x, weights, means, variances, n_iters, loglik_hist, ws, var_floor=1e-6,
                     stream=None):
    """gmm_fit with the screened-precision E-step (gmm_estep_accumulate_screened)."""
    gmm_fit(x, weights, means, variances, n_iters, loglik_hist, ws, var_floor, stream,
            _fn="gmm_fit_screened")


def gmm_assign_topk(x, weights, means, variances, m, tau, idx, resp, ws, stream=None):
    """Top-m multi-assignment into idx (int32 [n, m]) and resp (fp32 [n, m])."""
    import torch
    _dev(x, torch.float32, "x")
    n, d = x.shape
    k = weights.shape[0]
    rc = load_library().gmm_assign_topk(
        _ptr(x), n, d, k, _ptr(_dev(weights, torch.float32, "weights", k)),
        _ptr(_dev(means, torch.float32, "means", k * d)),
        _ptr(_dev(variances, torch.float32, "vars", k * d)),
        int(m), float(tau), _ptr(_dev(idx, torch.int32, "idx", n * m)),
        _ptr(_dev(resp, torch.float32, "resp", n * m)), _ptr(ws),
        ws.numel() if ws is not None else 0, _stream(stream))
    _check("gmm_assign_topk", rc)


def gmm_kmeans(x, weights, means, variances, n_iters, assign, ws, var_floor=1e-6, stream=None):
    """k-means warm start: n_iters Lloyd iterations on the centres in `means`, then the
    hard-assignment mixture into weights / means / variances (fp32 CUDA tensors, updated in
    place) and the last assignment into assign (int32 [n]).  ws: gmm.workspace(n, d, k, 1)."""
    import torch
    _dev(x, torch.float32, "x")
    n, d = x.shape
    k = weights.shape[0]
    rc = load_library().gmm_kmeans(
        _ptr(x), n, d, k, int(n_iters), float(var_floor),
        _ptr(_dev(weights, torch.float32, "weights", k)),
        _ptr(_dev(means, torch.float32, "means", k * d)),
        _ptr(_dev(variances, torch.float32, "vars", k * d)),
        _ptr(_dev(assign, torch.int32, "assign", n)), _ptr(ws),
        ws.numel() if ws is not None else 0, _stream(stream))
    _check("gmm_kmeans", rc)


def gmm_kmeanspp(x, u, idx, centers, ws=None, stream=None):
    """k-means++ seeding of k = u.numel() rows of x with the uniforms u (fp64 CUDA tensor,
    0 <= u < 1): chosen rows into idx (int64 [k]), their coordinates into centers (fp32
    [k, d]).  ws: a uint8 CUDA workspace (allocated here when None)."""
    import torch
    _dev(x, torch.float32, "x")
    n, d = x.shape
    k = u.numel()
    nb = load_library().gmm_kmeanspp_workspace_bytes(n)
    if ws is None:
        ws = torch.empty(nb, dtype=torch.uint8, device=x.device)
    rc = load_library().gmm_kmeanspp(
        _ptr(x), n, d, k, _ptr(_dev(u, torch.float64, "u", k)),
        _ptr(_dev(idx, torch.int64, "idx", k)), _ptr(_dev(centers, torch.float32, "centers", k * d)),
        _ptr(ws), ws.numel(), _stream(stream))
    _check("gmm_kmeanspp", rc)


def gmm_estep_accumulate_streamed(x_host, weights, means, variances, nk, s, q, loglik,
                                  chunk_rows, staging, ws, stream=None, copy_stream=None):
    """E-step of data held in page-locked host memory (x_host: a pinned fp32 CPU tensor
    [n, d]), uploaded chunk_rows rows at a time into `staging` (fp32 CUDA tensor of at least
    2 * min(chunk_rows, n) * d elements) on copy_stream while the previous chunk's E-step
    runs on `stream`; adds into nk, s, q, loglik as gmm_estep_accumulate does."""
    import torch
    if not (isinstance(x_host, torch.Tensor) and not x_host.is_cuda and x_host.is_pinned()
            and x_host.dtype == torch.float32 and x_host.is_contiguous() and x_host.dim() == 2):
        raise TypeError("x_host must be a contiguous pinned fp32 CPU tensor [n, d]")
    n, d = x_host.shape
    k = weights.shape[0]
    rows = min(int(chunk_rows), n) if chunk_rows >= 1 else 0
    rc = load_library().gmm_estep_accumulate_streamed(
        ctypes.c_void_p(x_host.data_ptr()), n, d, k,
        _ptr(_dev(weights, torch.float32, "weights", k)),
        _ptr(_dev(means, torch.float32, "means", k * d)),
        _ptr(_dev(variances, torch.float32, "vars", k * d)),
        _ptr(_dev(nk, torch.float64, "nk", k)), _ptr(_dev(s, torch.float64, "s", k * d)),
        _ptr(_dev(q, torch.float64, "q", k * d)), _ptr(_dev(loglik, torch.float64, "loglik", 1)),
        int(chunk_rows), _ptr(_dev(staging, torch.float32, "staging", 2 * rows * d)), _ptr(ws),
        ws.numel() if ws is not None else 0, _stream(stream), _stream(copy_stream))
    _check("gmm_estep_accumulate_streamed", rc)


# the C type of a ring's row source: fill(user, row0, rows, d, dst) -> 0 on success
FILL_FN = ctypes.CFUNCTYPE(ctypes.c_int, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64,
                           ctypes.c_int32, ctypes.c_void_p)


def gmm_estep_accumulate_ring(source, n, weights, means, variances, nk, s, q, loglik,
                              chunk_rows, ring, staging, ws, stream=None, copy_stream=None):
    """Out-of-core E-step whose rows come through a ring of page-locked staging chunks.

    source: a C-contiguous fp32 numpy array [n, d] in ordinary host memory (copied into
    the ring by the library's gmm_fill_pageable), or a callable fill(row0, rows, out) that
    writes rows row0 .. row0 + rows - 1 into the numpy view out [rows, d] of a ring slot.
    ring: a pinned fp32 CPU tensor [slots, min(chunk_rows, n), d] with slots >= 2; staging:
    an fp32 CUDA tensor of at least 2 * min(chunk_rows, n) * d elements.  Adds into nk, s,
    q, loglik as gmm_estep_accumulate does.  An exception raised by the callable ends the
    call (GMM_ERR_FILL) and is re-raised here."""
    import numpy as np
    import torch
    k = weights.shape[0]
    if not (isinstance(ring, torch.Tensor) and not ring.is_cuda and ring.is_pinned()
            and ring.dtype == torch.float32 and ring.is_contiguous() and ring.dim() == 3):
        raise TypeError("ring must be a contiguous pinned fp32 CPU tensor [slots, rows, d]")
    slots, rows, d = ring.shape
    if rows != min(int(chunk_rows), int(n)):
        raise ValueError(f"ring holds {rows} rows a slot, chunks are {min(int(chunk_rows), n)}")
    lib = load_library()
    failure = []
    if isinstance(source, np.ndarray):
        if not (source.dtype == np.float32 and source.flags.c_contiguous
                and source.shape == (n, d)):
            raise TypeError(f"source must be a C-contiguous float32 array [{n}, {d}]")
        fn = ctypes.cast(lib.gmm_fill_pageable, ctypes.c_void_p)
        user = ctypes.c_void_p(source.ctypes.data)
    elif callable(source):
        def trampoline(_user, row0, cnt, dd, dst):
            try:
                buf = (ctypes.c_float * (cnt * dd)).from_address(dst)
                source(int(row0), int(cnt), np.ctypeslib.as_array(buf).reshape(cnt, dd))
                return 0
            except BaseException as e:        # noqa: BLE001 - re-raised after the call
                failure.append(e)
                return 1
        cb = FILL_FN(trampoline)
        fn = ctypes.cast(cb, ctypes.c_void_p)
        user = ctypes.c_void_p(0)
    else:
        raise TypeError("source must be a numpy array or a callable")
    rc = lib.gmm_estep_accumulate_ring(
        fn, user, int(n), d, k,
        _ptr(_dev(weights, torch.float32, "weights", k)),
        _ptr(_dev(means, torch.float32, "means", k * d)),
        _ptr(_dev(variances, torch.float32, "vars", k * d)),
        _ptr(_dev(nk, torch.float64, "nk", k)), _ptr(_dev(s, torch.float64, "s", k * d)),
        _ptr(_dev(q, torch.float64, "q", k * d)), _ptr(_dev(loglik, torch.float64, "loglik", 1)),
        int(chunk_rows), ctypes.c_void_p(ring.data_ptr()), slots,
        _ptr(_dev(staging, torch.float32, "staging", 2 * rows * d)), _ptr(ws),
        ws.numel() if ws is not None else 0, _stream(stream), _stream(copy_stream))
    if failure:
        raise failure[0]
    _check("gmm_estep_accumulate_ring", rc)


def gmm_estep_accumulate_iso(x, weights, means, variances, nk, s, q, loglik, ws, stream=None):
    """Isotropic E-step (one variance per component, variances [k]): adds nk, s and the
    scalar q[k] = sum r ||x||^2 (fp64 CUDA tensors) and loglik."""
    import torch
    _dev(x, torch.float32, "x")
    n, d = x.shape
    k = weights.shape[0]
    rc = load_library().gmm_estep_accumulate_iso(
        _ptr(x), n, d, k, _ptr(_dev(weights, torch.float32, "weights", k)),
        _ptr(_dev(means, torch.float32, "means", k * d)),
        _ptr(_dev(variances, torch.float32, "vars", k)),
        _ptr(_dev(nk, torch.float64, "nk", k)), _ptr(_dev(s, torch.float64, "s", k * d)),
        _ptr(_dev(q, torch.float64, "q", k)), _ptr(_dev(loglik, torch.float64, "loglik", 1)),
        _ptr(ws), ws.numel() if ws is not None else 0, _stream(stream))
    _check("gmm_estep_accumulate_iso", rc)


def gmm_mstep_iso(nk, s, q, n_total, weights, means, variances, var_floor=1e-6, stream=None):
    """Isotropic M-step from fp64 statistics (q[k] scalar); updates the fp32 parameters."""
    import torch
    k, d = means.shape
    rc = load_library().gmm_mstep_iso(
        _ptr(_dev(nk, torch.float64, "nk", k)), _ptr(_dev(s, torch.float64, "s", k * d)),
        _ptr(_dev(q, torch.float64, "q", k)), float(n_total), d, k, float(var_floor),
        _ptr(_dev(weights, torch.float32, "weights", k)),
        _ptr(_dev(means, torch.float32, "means", k * d)),
        _ptr(_dev(variances, torch.float32, "vars", k)), _stream(stream))
    _check("gmm_mstep_iso", rc)


def gmm_fit_iso(x, weights, means, variances, n_iters, loglik_hist, ws, var_floor=1e-6,
                stream=None):
    """n_iters isotropic EM iterations (variances [k]); loglik_hist[t] = LL(Theta_t)."""
    import torch
    _dev(x, torch.float32, "x")
    n, d = x.shape
    k = weights.shape[0]
    rc = load_library().gmm_fit_iso(
        _ptr(x), n, d, k, int(n_iters), float(var_floor),
        _ptr(_dev(weights, torch.float32, "weights", k)),
        _ptr(_dev(means, torch.float32, "means", k * d)),
        _ptr(_dev(variances, torch.float32, "vars", k)),
        _ptr(_dev(loglik_hist, torch.float64, "loglik_hist", n_iters)), _ptr(ws),
        ws.numel() if ws is not None else 0, _stream(stream))
    _check("gmm_fit_iso", rc)


TIMING_PHASES = ("prep", "logz", "exact_pairs", "dense_stats", "ill_light_and_reduce")


def gmm_timing_enable(on: bool = True):
    """Switches the E-step phase timing on or off and zeroes its totals."""
    _check("gmm_timing_enable", load_library().gmm_timing_enable(1 if on else 0))


def gmm_timing_read():
    """(dict phase -> total GPU ms, number of timed E-steps) since gmm_timing_enable."""
    ms = (ctypes.c_double * len(TIMING_PHASES))()
    calls = ctypes.c_int64(0)
    _check("gmm_timing_read", load_library().gmm_timing_read(
        ctypes.cast(ms, ctypes.c_void_p), len(TIMING_PHASES),
        ctypes.cast(ctypes.byref(calls), ctypes.c_void_p)))
    return dict(zip(TIMING_PHASES, list(ms))), calls.value


def gmm_set_stats_chunk_limit(max_chunks: int = 0):
    """Caps the point chunks of the dense statistics pass (0: the automatic count).
    Process-wide; results change by rounding only."""
    _check("gmm_set_stats_chunk_limit", load_library().gmm_set_stats_chunk_limit(int(max_chunks)))


def gmm_estep_accumulate_static(x, weights, means, variances, nk, s, q, loglik, stream=None):
    """gmm_estep_accumulate with the library's own static device workspace (no workspace
    argument, nothing allocated); raises GMMError(GMM_ERR_WORKSPACE) for shapes it cannot
    hold."""
    import torch
    _dev(x, torch.float32, "x")
    n, d = x.shape
    k = weights.shape[0]
    rc = load_library().gmm_estep_accumulate_static(
        _ptr(x), n, d, k, _ptr(_dev(weights, torch.float32, "weights", k)),
        _ptr(_dev(means, torch.float32, "means", k * d)),
        _ptr(_dev(variances, torch.float32, "vars", k * d)),
        _ptr(_dev(nk, torch.float64, "nk", k)), _ptr(_dev(s, torch.float64, "s", k * d)),
        _ptr(_dev(q, torch.float64, "q", k * d)), _ptr(_dev(loglik, torch.float64, "loglik", 1)),
        _stream(stream))
    _check("gmm_estep_accumulate_static", rc)
