"""Seeded synthetic workloads for the diagonal-GMM EM hot path.

This package only draws inputs: the data matrix X, the true mixture it comes
from, and the random-point initial parameters.  It holds none of the EM
arithmetic, so both the GPU path and the CPU checker can use it without
sharing any of the method's code.

The shapes follow the paper's runtime study (Table 1: K=1024 components,
D=128, N from 1e4 to 1e8) and its IVF use case (Sec. 4, unit-normalised
embedding-like vectors).  The paper does not say which data its runtime
table used, so these generators stand in for it; the IVF datasets it
evaluates on are replaced by unit-normalised samples of anisotropic diagonal
Gaussians.

All draws come from Philox4x32-10 (see ``synth.c``); any row slice of X can
be regenerated on its own, bit for bit.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libsynth.so")
_lib = None


def build_lib(force: bool = True) -> str:
    """Compile ``synth.c`` into ``libsynth.so`` next to it (gcc, -O2)."""
    src = os.path.join(_HERE, "synth.c")
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
        c_dp = ctypes.POINTER(ctypes.c_double)
        lib.synth_true_mixture.argtypes = [ctypes.c_uint64, ctypes.c_int32, ctypes.c_int32,
                                           ctypes.c_double, ctypes.c_double, ctypes.c_double,
                                           c_dp, c_dp, c_dp]
        lib.synth_true_mixture.restype = None
        lib.synth_rows.argtypes = [ctypes.c_uint64, ctypes.c_int64, ctypes.c_int64, ctypes.c_int32,
                                   ctypes.c_int32, c_dp, c_dp, c_dp, ctypes.c_int32, ctypes.c_int32,
                                   ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                                   ctypes.c_void_p]
        lib.synth_rows.restype = ctypes.c_int
        lib.synth_init_rows.argtypes = [ctypes.c_uint64, ctypes.c_int64, ctypes.c_int32,
                                        ctypes.c_void_p]
        lib.synth_init_rows.restype = ctypes.c_int
        lib.synth_philox4x32_10.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
        lib.synth_philox4x32_10.restype = None
        _lib = lib
    return _lib


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.c_void_p)


def _dptr(a: np.ndarray):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def philox4x32_10(counter, key) -> np.ndarray:
    """One Philox4x32-10 block: four 32-bit outputs for a 4-word counter and 2-word key."""
    c = np.ascontiguousarray(counter, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    out = np.zeros(4, dtype=np.uint32)
    _load().synth_philox4x32_10(_ptr(c), _ptr(k), _ptr(out))
    return out


@dataclasses.dataclass(frozen=True)
class Workload:
    """One synthetic EM workload (data recipe + fit settings)."""
    name: str
    n: int              # points
    d: int              # dimensions
    k_true: int         # components the data is drawn from
    k: int              # components fitted
    iters: int          # EM iterations
    data_seed: int
    init_seed: int
    normalize: bool = False   # unit-normalise each row (IVF-style embeddings)
    assign_m: int = 0         # top-m multi-assignment after the fit (0 = none)
    mean_std: float = 2.0     # true means ~ N(0, mean_std^2)
    std_lo: float = 0.5       # true per-dim std ~ U[std_lo, std_hi]
    std_hi: float = 1.5

    @property
    def tau(self) -> float:
        """Multi-assignment threshold: the uniform prior 1/K (paper Sec. 4.3)."""
        return 1.0 / self.k


WORKLOADS = {
    "tiny": Workload("tiny", 10_000, 16, 8, 8, 10, 1, 1001),
    "small": Workload("small", 100_000, 128, 1024, 1024, 30, 2, 1002),
    "mid": Workload("mid", 1_000_000, 128, 1024, 1024, 30, 3, 1003),
    "large": Workload("large", 100_000_000, 128, 1024, 1024, 30, 4, 1004),
    "ivf": Workload("ivf", 5_000_000, 768, 8192, 4096, 20, 5, 1005, normalize=True, assign_m=2),
}


def custom(name: str, n: int, d: int, k_true: int, k: int, iters: int = 1, data_seed: int = 7,
           init_seed: int = 1007, normalize: bool = False) -> Workload:
    """A workload of arbitrary shape with the same generator (tests use these)."""
    return Workload(name, n, d, k_true, k, iters, data_seed, init_seed, normalize)


class Mixture:
    """The true mixture of a workload, fp64."""

    def __init__(self, w: Workload):
        self.w = w
        self.means = np.zeros((w.k_true, w.d), dtype=np.float64)
        self.stds = np.zeros((w.k_true, w.d), dtype=np.float64)
        self.weights = np.zeros(w.k_true, dtype=np.float64)
        _load().synth_true_mixture(w.data_seed, w.k_true, w.d, w.mean_std, w.std_lo, w.std_hi,
                                   _dptr(self.means), _dptr(self.stds), _dptr(self.weights))

    def rows(self, row0: int, row1: int, out: np.ndarray | None = None, nthreads: int | None = None,
             want_comp: bool = False, want_colstats: bool = False):
        """Rows [row0, row1) of X as fp32 (row1-row0, d); optionally the true components and
        fp64 column sums / sums of squares of the slice."""
        w = self.w
        n = row1 - row0
        if out is None:
            out = np.empty((n, w.d), dtype=np.float32)
        assert out.dtype == np.float32 and out.flags.c_contiguous and out.shape == (n, w.d)
        comp = np.empty(n, dtype=np.int32) if want_comp else None
        cs = np.empty(w.d, dtype=np.float64) if want_colstats else None
        cq = np.empty(w.d, dtype=np.float64) if want_colstats else None
        nt = nthreads or min(16, os.cpu_count() or 1)
        rc = _load().synth_rows(w.data_seed, row0, row1, w.d, w.k_true, _dptr(self.means),
                                _dptr(self.stds), _dptr(self.weights), int(w.normalize), nt,
                                _ptr(out), _ptr(comp) if comp is not None else None,
                                _ptr(cs) if cs is not None else None,
                                _ptr(cq) if cq is not None else None)
        if rc != 0:
            raise ValueError("synth_rows failed")
        res = [out]
        if want_comp:
            res.append(comp)
        if want_colstats:
            res += [cs, cq]
        return res[0] if len(res) == 1 else tuple(res)


def init_rows(w: Workload) -> np.ndarray:
    """K distinct row indices for the random-point initialisation."""
    rows = np.empty(w.k, dtype=np.int64)
    if _load().synth_init_rows(w.init_seed, w.n, w.k, _ptr(rows)) != 0:
        raise ValueError("need n >= k for random-point init")
    return rows


def random_point_init(w: Workload, mix: Mixture, colsum: np.ndarray, colsq: np.ndarray):
    """Random-point initial parameters (fp32): means = K distinct data rows, every component's
    variance = the global per-dim population variance of X (divide by N, computed in fp64 from
    the column sums), weights = 1/K.  Returns (weights[K], means[K,D], vars[K,D])."""
    rows = init_rows(w)
    means = np.empty((w.k, w.d), dtype=np.float32)
    for j, r in enumerate(rows):
        means[j] = mix.rows(int(r), int(r) + 1, nthreads=1)[0]
    mean = colsum / w.n
    var = np.maximum(colsq / w.n - mean * mean, 0.0)
    variances = np.broadcast_to(var.astype(np.float32), (w.k, w.d)).copy()
    weights = np.full(w.k, 1.0 / w.k, dtype=np.float32)
    return weights, means, variances


def make(w: Workload | str, nthreads: int | None = None):
    """Whole workload in host memory: (X fp32 [N,D], (weights, means, vars) fp32 init)."""
    if isinstance(w, str):
        w = WORKLOADS[w]
    mix = Mixture(w)
    x, cs, cq = mix.rows(0, w.n, nthreads=nthreads, want_colstats=True)
    return x, random_point_init(w, mix, cs, cq)
