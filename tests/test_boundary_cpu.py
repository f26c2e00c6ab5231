"""The C ABI without a GPU: the library loads, exports every symbol the header
declares, sizes its workspace, and rejects bad arguments on the host before
enqueuing anything."""
import ctypes
import os
import re

import pytest

import paper_2606_10896_amd as gmm

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _header_functions():
    src = open(os.path.join(ROOT, "include", "flashgmm.h")).read()
    return sorted(set(re.findall(r"^(?:const char\*|size_t|int)\s+(gmm_\w+)\(", src, re.M)))


def test_library_exports_every_declared_symbol():
    lib = gmm.load_library()
    names = _header_functions()
    assert set(names) == set(gmm.EXPORTS)
    for name in names:
        assert getattr(lib, name) is not None


def test_status_strings():
    assert gmm.status_string(0) == "GMM_OK"
    assert gmm.status_string(-1) == "GMM_ERR_INVALID_ARG"
    assert gmm.status_string(-2) == "GMM_ERR_UNSUPPORTED"
    assert gmm.status_string(-3) == "GMM_ERR_WORKSPACE"
    assert gmm.status_string(-4) == "GMM_ERR_DEVICE"
    assert gmm.status_string(-5) == "GMM_ERR_FILL"
    assert gmm.status_string(12345) == "GMM_UNKNOWN_STATUS"


@pytest.mark.parametrize("n,d,k", [(1, 1, 1), (10_000, 16, 8), (100_000, 128, 1024),
                                   (100_000_000, 128, 1024), (1_000_003, 37, 45),
                                   (5_000, 256, 65535), (5_000_000, 768, 4096), (1_000, 1024, 64),
                                   (3_000, 300, 17)])
def test_workspace_is_o_n_plus_o_kd(n, d, k):
    nb = gmm.workspace_bytes(n, d, k)
    assert nb > 0 and nb % 256 == 0
    # per point: one fp64 log-normaliser, 4 refined (16-bit slot, fp32 responsibility) pairs,
    # room for 4 bucketed pair records (16 B each), a 64-bit mask of the component blocks
    # the dense statistics take (k <= 4096), a flag byte for the routed components and at most
    # 1/4 of an fp64 log-likelihood partial; plus O(k d) parameters and partial statistics:
    # never n x k
    assert nb >= 96 * n
    dp = (d + 63) // 64 * 64 if d <= 256 else (d + 127) // 128 * 128
    kpad = (k + 63) // 64 * 64
    row = 8 * (1 + 2 * dp)
    well_part = row * max(8 * kpad, 8192 * 64)
    sparse_part = row * max(kpad, 8192 * 32)
    ill_part = row * max(kpad + 32, 512 * 32)
    # the routed components' partials, and as many for the exact recomputation of the light
    # components (plus their flags, list positions and list: 9 bytes per component)
    okd = well_part + sparse_part + 2 * ill_part + 40 * kpad * dp + 8 * 2 * k * d + 9 * k
    # + two flag bytes: a routed component, a light component holds mass at the point
    per_pt = (104 if kpad <= 4096 else 96) + 2
    assert nb <= per_pt * n + n // 4 + okd + 64 * k + (4 << 20)
    if n >= 10 ** 6 and k >= 1024:
        # a small fraction of what an n x k fp32 responsibility array would take
        assert nb < n * k * 4 / 25


@pytest.mark.parametrize("n,d,k,m", [(0, 8, 4, 0), (10, 0, 4, 0), (10, 8, 0, 0), (10, 1025, 4, 0),
                                     (10, 8, 65536, 0), (10, 8, 4, 9), (10, 8, 4, -1)])
def test_workspace_rejects_bad_shapes(n, d, k, m):
    assert gmm.workspace_bytes(n, d, k, m) == 0


def _fake(addr=0x100000):
    return ctypes.c_void_p(addr)


def test_host_validation_returns_before_any_launch():
    lib = gmm.load_library()
    p, ws = _fake(), _fake(0x200000)
    big = gmm.workspace_bytes(1000, 8, 4)
    # non-positive sizes and null pointers
    assert lib.gmm_estep_accumulate(p, 0, 8, 4, p, p, p, p, p, p, p, ws, big, None) == gmm.GMM_ERR_INVALID_ARG
    assert lib.gmm_estep_accumulate(p, 1000, 8, 4, None, p, p, p, p, p, p, ws, big, None) == gmm.GMM_ERR_INVALID_ARG
    assert lib.gmm_estep_accumulate(p, 1000, 1025, 4, p, p, p, p, p, p, p, ws, big, None) == gmm.GMM_ERR_UNSUPPORTED
    # workspace: missing, misaligned, too small
    assert lib.gmm_estep_accumulate(p, 1000, 8, 4, p, p, p, p, p, p, p, None, big, None) == gmm.GMM_ERR_WORKSPACE
    assert lib.gmm_estep_accumulate(p, 1000, 8, 4, p, p, p, p, p, p, p, _fake(0x200010), big, None) == gmm.GMM_ERR_WORKSPACE
    assert lib.gmm_estep_accumulate(p, 1000, 8, 4, p, p, p, p, p, p, p, ws, big - 1, None) == gmm.GMM_ERR_WORKSPACE
    assert lib.gmm_fit(p, 1000, 8, 4, -1, 1e-6, p, p, p, p, ws, big, None) == gmm.GMM_ERR_INVALID_ARG
    assert lib.gmm_fit(p, 1000, 8, 4, 3, -1.0, p, p, p, p, ws, big, None) == gmm.GMM_ERR_INVALID_ARG
    assert lib.gmm_fit(p, 1000, 8, 4, 3, 1e-6, p, p, p, None, ws, big, None) == gmm.GMM_ERR_INVALID_ARG
    assert lib.gmm_mstep(p, p, p, 0.0, 8, 4, 1e-6, p, p, p, None) == gmm.GMM_ERR_INVALID_ARG
    assert lib.gmm_mstep(p, p, p, 10.0, 8, 4, -1.0, p, p, p, None) == gmm.GMM_ERR_INVALID_ARG
    assert lib.gmm_mstep(None, p, p, 10.0, 8, 4, 1e-6, p, p, p, None) == gmm.GMM_ERR_INVALID_ARG


def test_isotropic_host_validation():
    lib = gmm.load_library()
    p, ws = _fake(), _fake(0x200000)
    big = gmm.workspace_bytes(1000, 8, 4)
    assert lib.gmm_estep_accumulate_iso(p, 0, 8, 4, p, p, p, p, p, p, p, ws, big, None) == gmm.GMM_ERR_INVALID_ARG
    assert lib.gmm_estep_accumulate_iso(p, 1000, 8, 4, p, p, None, p, p, p, p, ws, big, None) == gmm.GMM_ERR_INVALID_ARG
    assert lib.gmm_estep_accumulate_iso(p, 1000, 1025, 4, p, p, p, p, p, p, p, ws, big, None) == gmm.GMM_ERR_UNSUPPORTED
    assert lib.gmm_estep_accumulate_iso(p, 1000, 8, 4, p, p, p, p, p, p, p, ws, big - 1, None) == gmm.GMM_ERR_WORKSPACE
    assert lib.gmm_fit_iso(p, 1000, 8, 4, -1, 1e-6, p, p, p, p, ws, big, None) == gmm.GMM_ERR_INVALID_ARG
    assert lib.gmm_fit_iso(p, 1000, 8, 4, 3, 1e-6, p, p, p, None, ws, big, None) == gmm.GMM_ERR_INVALID_ARG
    assert lib.gmm_fit_iso(p, 1000, 8, 4, 3, 1e-6, p, p, p, p, None, big, None) == gmm.GMM_ERR_WORKSPACE
    assert lib.gmm_mstep_iso(p, p, p, 0.0, 8, 4, 1e-6, p, p, p, None) == gmm.GMM_ERR_INVALID_ARG
    assert lib.gmm_mstep_iso(p, p, None, 10.0, 8, 4, 1e-6, p, p, p, None) == gmm.GMM_ERR_INVALID_ARG
    assert lib.gmm_mstep_iso(p, p, p, 10.0, 1025, 4, 1e-6, p, p, p, None) == gmm.GMM_ERR_UNSUPPORTED


def test_screened_host_validation():
    """The reduced-precision calls validate their arguments as the exact ones do."""
    lib = gmm.load_library()
    p, ws = _fake(), _fake(0x200000)
    big = gmm.workspace_bytes(1000, 8, 4)
    e = lib.gmm_estep_accumulate_screened
    assert e(p, 0, 8, 4, p, p, p, p, p, p, p, ws, big, None) == gmm.GMM_ERR_INVALID_ARG
    assert e(p, 1000, 8, 4, None, p, p, p, p, p, p, ws, big, None) == gmm.GMM_ERR_INVALID_ARG
    assert e(p, 1000, 1025, 4, p, p, p, p, p, p, p, ws, big, None) == gmm.GMM_ERR_UNSUPPORTED
    assert e(p, 1000, 8, 4, p, p, p, p, p, p, p, ws, big - 1, None) == gmm.GMM_ERR_WORKSPACE
    f = lib.gmm_fit_screened
    assert f(p, 1000, 8, 4, -1, 1e-6, p, p, p, p, ws, big, None) == gmm.GMM_ERR_INVALID_ARG
    assert f(p, 1000, 8, 4, 3, -1.0, p, p, p, p, ws, big, None) == gmm.GMM_ERR_INVALID_ARG
    assert f(p, 1000, 8, 4, 3, 1e-6, p, p, p, None, ws, big, None) == gmm.GMM_ERR_INVALID_ARG
    assert f(p, 1000, 8, 4, 3, 1e-6, p, p, p, p, None, big, None) == gmm.GMM_ERR_WORKSPACE


def test_streamed_host_validation():
    lib = gmm.load_library()
    p, ws = _fake(), _fake(0x200000)
    small = gmm.workspace_bytes(500, 8, 4)
    call = lambda xh, chunk, stg, w, nb: lib.gmm_estep_accumulate_streamed(
        xh, 1000, 8, 4, p, p, p, p, p, p, p, chunk, stg, w, nb, None, None)
    assert call(None, 500, p, ws, small) == gmm.GMM_ERR_INVALID_ARG
    assert call(p, 0, p, ws, small) == gmm.GMM_ERR_INVALID_ARG
    assert call(p, 500, None, ws, small) == gmm.GMM_ERR_INVALID_ARG
    # the workspace is sized for one chunk of min(chunk_rows, n) rows
    assert call(p, 500, p, ws, small - 1) == gmm.GMM_ERR_WORKSPACE
    assert call(p, 5000, p, ws, small) == gmm.GMM_ERR_WORKSPACE
    assert lib.gmm_estep_accumulate_streamed(p, 1000, 1025, 4, p, p, p, p, p, p, p, 500, p, ws,
                                             small, None, None) == gmm.GMM_ERR_UNSUPPORTED


def test_ring_host_validation():
    lib = gmm.load_library()
    p, ws = _fake(), _fake(0x200000)
    fill = ctypes.cast(lib.gmm_fill_pageable, ctypes.c_void_p)
    small = gmm.workspace_bytes(500, 8, 4)
    call = lambda fn, chunk, ring, slots, stg, w, nb: lib.gmm_estep_accumulate_ring(
        fn, p, 1000, 8, 4, p, p, p, p, p, p, p, chunk, ring, slots, stg, w, nb, None, None)
    assert call(None, 500, p, 2, p, ws, small) == gmm.GMM_ERR_INVALID_ARG
    assert call(fill, 0, p, 2, p, ws, small) == gmm.GMM_ERR_INVALID_ARG
    assert call(fill, 500, None, 2, p, ws, small) == gmm.GMM_ERR_INVALID_ARG
    assert call(fill, 500, p, 1, p, ws, small) == gmm.GMM_ERR_INVALID_ARG
    assert call(fill, 500, p, 2, None, ws, small) == gmm.GMM_ERR_INVALID_ARG
    # the workspace is sized for one chunk of min(chunk_rows, n) rows
    assert call(fill, 500, p, 2, p, ws, small - 1) == gmm.GMM_ERR_WORKSPACE
    assert call(fill, 5000, p, 3, p, ws, small) == gmm.GMM_ERR_WORKSPACE
    assert lib.gmm_estep_accumulate_ring(fill, p, 1000, 1025, 4, p, p, p, p, p, p, p, 500, p, 2,
                                         p, ws, small, None, None) == gmm.GMM_ERR_UNSUPPORTED


@pytest.mark.parametrize("n,d,row0,rows", [(1000, 7, 0, 1000), (1000, 7, 993, 7), (1000, 7, 10, 0),
                                           (170_000, 128, 3, 169_990)])
def test_fill_pageable_copies_the_rows(n, d, row0, rows):
    """The pageable-memory row source is plain host code: rows row0 .. row0 + rows - 1, whole,
    also when the copy is split over threads (above 64 MiB: the last case, 87 MB)."""
    import numpy as np
    lib = gmm.load_library()
    x = np.random.default_rng(n + row0).standard_normal((n, d)).astype(np.float32)
    out = np.full((max(rows, 1) + 1, d), np.float32(-7.0))
    rc = lib.gmm_fill_pageable(ctypes.c_void_p(x.ctypes.data), row0, rows, d,
                               ctypes.c_void_p(out.ctypes.data))
    assert rc == 0
    np.testing.assert_array_equal(out[:rows], x[row0:row0 + rows])
    assert np.all(out[rows:] == np.float32(-7.0))
    assert lib.gmm_fill_pageable(None, 0, 1, d, ctypes.c_void_p(out.ctypes.data)) == 1
    assert lib.gmm_fill_pageable(ctypes.c_void_p(x.ctypes.data), 0, -1, d,
                                 ctypes.c_void_p(out.ctypes.data)) == 1


def test_kmeanspp_host_validation():
    lib = gmm.load_library()
    p, ws = _fake(), _fake(0x200000)
    nb = lib.gmm_kmeanspp_workspace_bytes(10000)
    assert nb >= 8 * 10000 and nb % 256 == 0 and lib.gmm_kmeanspp_workspace_bytes(0) == 0
    assert lib.gmm_kmeanspp(None, 10000, 8, 4, p, p, p, ws, nb, None) == gmm.GMM_ERR_INVALID_ARG
    assert lib.gmm_kmeanspp(p, 10000, 8, 4, None, p, p, ws, nb, None) == gmm.GMM_ERR_INVALID_ARG
    assert lib.gmm_kmeanspp(p, 0, 8, 4, p, p, p, ws, nb, None) == gmm.GMM_ERR_INVALID_ARG
    assert lib.gmm_kmeanspp(p, 10000, 1025, 4, p, p, p, ws, nb, None) == gmm.GMM_ERR_UNSUPPORTED
    assert lib.gmm_kmeanspp(p, 10000, 8, 4, p, p, p, ws, nb - 1, None) == gmm.GMM_ERR_WORKSPACE
    assert lib.gmm_kmeanspp(p, 10000, 8, 4, p, p, p, _fake(0x200008), nb, None) == gmm.GMM_ERR_WORKSPACE


def test_kmeans_host_validation():
    lib = gmm.load_library()
    p, ws = _fake(), _fake(0x200000)
    nb = gmm.workspace_bytes(1000, 8, 4, 1)
    assert lib.gmm_kmeans(p, 1000, 8, 4, -1, 1e-6, p, p, p, p, ws, nb, None) == gmm.GMM_ERR_INVALID_ARG
    assert lib.gmm_kmeans(p, 1000, 8, 4, 3, -1.0, p, p, p, p, ws, nb, None) == gmm.GMM_ERR_INVALID_ARG
    assert lib.gmm_kmeans(p, 1000, 8, 4, 3, 1e-6, p, p, p, None, ws, nb, None) == gmm.GMM_ERR_INVALID_ARG
    assert lib.gmm_kmeans(p, 1000, 1025, 4, 3, 1e-6, p, p, p, p, ws, nb, None) == gmm.GMM_ERR_UNSUPPORTED
    assert lib.gmm_kmeans(p, 1000, 8, 4, 3, 1e-6, p, p, p, p, ws, nb - 1, None) == gmm.GMM_ERR_WORKSPACE


def test_assign_host_validation():
    lib = gmm.load_library()
    p, ws = _fake(), _fake(0x200000)
    big = gmm.workspace_bytes(1000, 8, 4, 2)
    call = lambda m, tau, **kw: lib.gmm_assign_topk(
        kw.get("x", p), kw.get("n", 1000), kw.get("d", 8), kw.get("k", 4), p, p, p, m,
        ctypes.c_float(tau), kw.get("idx", p), p, kw.get("ws", ws), kw.get("wsb", big), None)
    assert call(9, 0.1) == gmm.GMM_ERR_UNSUPPORTED            # m > GMM_MAX_M
    assert call(0, 0.1) == gmm.GMM_ERR_INVALID_ARG            # m < 1
    assert call(5, 0.1) == gmm.GMM_ERR_INVALID_ARG            # m > k
    assert call(2, -0.1) == gmm.GMM_ERR_INVALID_ARG           # tau < 0
    assert call(2, 1.0) == gmm.GMM_ERR_INVALID_ARG            # tau >= 1
    assert call(2, float("nan")) == gmm.GMM_ERR_INVALID_ARG
    assert call(2, 0.1, idx=None) == gmm.GMM_ERR_INVALID_ARG
    assert call(2, 0.1, d=1025) == gmm.GMM_ERR_UNSUPPORTED
    assert call(2, 0.1, n=0) == gmm.GMM_ERR_INVALID_ARG
    assert call(2, 0.1, ws=None) == gmm.GMM_ERR_WORKSPACE
    assert call(2, 0.1, wsb=big - 1) == gmm.GMM_ERR_WORKSPACE


def test_timing_switch_and_read_on_the_host():
    # switching off creates no events and needs no device; the totals read back as zeros
    lib = gmm.load_library()
    assert lib.gmm_timing_enable(0) == 0
    totals, calls = gmm.gmm_timing_read()
    assert calls == 0 and set(totals) == set(gmm.TIMING_PHASES)
    assert all(v == 0.0 for v in totals.values())
    assert lib.gmm_timing_read(None, 5, None) == -1
    ms = (ctypes.c_double * 7)(*([1.0] * 7))
    calls_c = ctypes.c_int64(5)
    assert lib.gmm_timing_read(ctypes.cast(ms, ctypes.c_void_p), 7,
                               ctypes.cast(ctypes.byref(calls_c), ctypes.c_void_p)) == 0
    assert list(ms) == [0.0] * 7 and calls_c.value == 0
    assert lib.gmm_timing_read(ctypes.cast(ms, ctypes.c_void_p), -1,
                               ctypes.cast(ctypes.byref(calls_c), ctypes.c_void_p)) == -1



def test_stats_chunk_limit_is_checked_and_never_grows_the_workspace():
    lib = gmm.load_library()
    assert lib.gmm_set_stats_chunk_limit(-1) == gmm.GMM_ERR_INVALID_ARG
    auto = gmm.workspace_bytes(1_000_000, 128, 1024)
    try:
        for cap in (1, 16, 100000):
            assert lib.gmm_set_stats_chunk_limit(cap) == gmm.GMM_OK
            assert 0 < gmm.workspace_bytes(1_000_000, 128, 1024) <= auto
        assert lib.gmm_set_stats_chunk_limit(1) == gmm.GMM_OK
        assert gmm.workspace_bytes(1_000_000, 128, 1024) < auto
    finally:
        assert lib.gmm_set_stats_chunk_limit(0) == gmm.GMM_OK
    assert gmm.workspace_bytes(1_000_000, 128, 1024) == auto


def test_static_estep_refuses_shapes_beyond_its_array_before_any_launch():
    """gmm_estep_accumulate_static: a shape whose workspace cannot fit the library's 64 MiB
    array is refused on the host (GMM_ERR_WORKSPACE), whatever the pointers; null pointers are
    invalid arguments."""
    lib = gmm.load_library()
    f = _fake()
    assert lib.gmm_estep_accumulate_static(f, 475_777, 128, 1024, f, f, f, f, f, f, f,
                                           None) == gmm.GMM_ERR_WORKSPACE
    assert lib.gmm_estep_accumulate_static(f, 1000, 768, 4096, f, f, f, f, f, f, f,
                                           None) == gmm.GMM_ERR_WORKSPACE
    assert lib.gmm_estep_accumulate_static(None, 1000, 16, 8, f, f, f, f, f, f, f,
                                           None) == gmm.GMM_ERR_INVALID_ARG
    assert lib.gmm_estep_accumulate_static(f, 0, 16, 8, f, f, f, f, f, f, f,
                                           None) == gmm.GMM_ERR_INVALID_ARG
