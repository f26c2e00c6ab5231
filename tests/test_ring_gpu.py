"""The out-of-core E-step over a ring of page-locked staging chunks: rows come from ordinary
host memory (the library's pageable-memory source) or from a caller's fill function, and the
statistics must equal, bit for bit, those of gmm_estep_accumulate called chunk by chunk on
device copies of the same rows, across EM iterations that reuse the ring, and match the
checker.  The 1e8-row case (X in pageable memory) is in test_large_fulln_gpu.py."""
import sys

import numpy as np
import pytest

import gmm_synth as g
import oracle
from gmmcheck import check_stats

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _zeros(k, d):
    import torch
    return (torch.zeros(k, dtype=torch.float64, device="cuda"),
            torch.zeros(k, d, dtype=torch.float64, device="cuda"),
            torch.zeros(k, d, dtype=torch.float64, device="cuda"),
            torch.zeros(1, dtype=torch.float64, device="cuda"))


def _buffers(n, d, k, chunk, slots):
    import torch
    import paper_2606_10896_amd as gmm
    rows = min(chunk, n)
    return (torch.empty((slots, rows, d), dtype=torch.float32, pin_memory=True),
            torch.empty(2 * rows * d, dtype=torch.float32, device="cuda"),
            gmm.workspace(rows, d, k), torch.cuda.Stream())


@pytest.mark.parametrize("n,d,kt,k,chunk,slots", [(50001, 128, 24, 64, 12000, 2),
                                                  (20000, 300, 10, 30, 7001, 3),
                                                  (9000, 40, 6, 9, 9000, 2),
                                                  (30000, 64, 8, 20, 2999, 4)])
def test_ring_equals_chunk_by_chunk_calls(n, d, kt, k, chunk, slots):
    import torch
    import paper_2606_10896_amd as gmm
    w = g.custom(f"ring{n}_{d}", n, d, kt, k, data_seed=7 + d, init_seed=8 + k)
    x, th0 = g.make(w)
    _say(f"  ring E-step n={n} d={d} k={k} chunk={chunk} slots={slots}")
    ring, staging, ws, copy = _buffers(n, d, k, chunk, slots)
    rows = min(chunk, n)
    chunks = [torch.from_numpy(x[r0:r0 + rows]).cuda() for r0 in range(0, n, rows)]
    ws_ref = gmm.workspace(rows, d, k)
    tha = [torch.from_numpy(a).cuda() for a in th0]
    thb = [torch.from_numpy(a).cuda() for a in th0]
    for it in range(3):
        a = _zeros(k, d)
        gmm.gmm_estep_accumulate_ring(x, n, *tha, *a, chunk, ring, staging, ws, copy_stream=copy)
        b = _zeros(k, d)
        for xc in chunks:
            gmm.gmm_estep_accumulate(xc, *thb, *b, ws_ref)
        torch.cuda.synchronize()
        for u, v in zip(a, b):
            assert torch.equal(u, v), f"iteration {it}: ring and chunked statistics differ"
        if it == 0:
            ref = oracle.estep(x, *th0)
            st = dict(nk=a[0].cpu().numpy(), s=a[1].cpu().numpy(), q=a[2].cpu().numpy(),
                      loglik=a[3].item())
            _say("  ", check_stats(st, ref, "ring t=0"))
        gmm.gmm_mstep(*a[:3], float(n), *tha)
        gmm.gmm_mstep(*b[:3], float(n), *thb)
    torch.cuda.synchronize()
    for u, v in zip(tha, thb):
        assert torch.equal(u, v)


def test_ring_fill_function_is_called_in_row_order():
    """A caller's fill function (here one that generates the rows on demand from the seeded
    generator, so X never exists whole in host memory) is called once per chunk, in row order,
    covering every row once; the statistics equal those of the pageable-memory source."""
    import torch
    import paper_2606_10896_amd as gmm
    w = g.custom("ringcb", 40000, 96, 12, 40, data_seed=31, init_seed=32)
    x, th0 = g.make(w)
    mix = g.Mixture(w)
    n, d, k, chunk = w.n, w.d, w.k, 6000
    calls = []

    def fill(row0, rows, out):
        calls.append((row0, rows))
        mix.rows(row0, row0 + rows, out=out, nthreads=4)

    ring, staging, ws, copy = _buffers(n, d, k, chunk, 3)
    th = [torch.from_numpy(a).cuda() for a in th0]
    a = _zeros(k, d)
    gmm.gmm_estep_accumulate_ring(fill, n, *th, *a, chunk, ring, staging, ws, copy_stream=copy)
    b = _zeros(k, d)
    gmm.gmm_estep_accumulate_ring(x, n, *th, *b, chunk, ring, staging, ws, copy_stream=copy)
    torch.cuda.synchronize()
    assert calls == [(r0, min(chunk, n - r0)) for r0 in range(0, n, chunk)]
    for u, v in zip(a, b):
        assert torch.equal(u, v)
    _say(f"  {len(calls)} fills in row order; generated rows equal the array's")


def test_ring_fill_failure_ends_the_call():
    """A fill function that fails ends the call with GMM_ERR_FILL (the binding re-raises the
    callable's exception) after the chunks before it were enqueued; the ring then serves the
    next call normally."""
    import torch
    import paper_2606_10896_amd as gmm
    w = g.custom("ringerr", 12000, 32, 6, 10, data_seed=41, init_seed=42)
    x, th0 = g.make(w)
    n, d, k, chunk = w.n, w.d, w.k, 2500

    def fill(row0, rows, out):
        if row0 >= 2 * chunk:
            raise ValueError("source exhausted")
        out[:] = x[row0:row0 + rows]

    ring, staging, ws, copy = _buffers(n, d, k, chunk, 2)
    th = [torch.from_numpy(a).cuda() for a in th0]
    a = _zeros(k, d)
    with pytest.raises(ValueError, match="source exhausted"):
        gmm.gmm_estep_accumulate_ring(fill, n, *th, *a, chunk, ring, staging, ws,
                                      copy_stream=copy)
    torch.cuda.synchronize()
    # the two chunks enqueued before the failure were added (a point's responsibilities sum
    # to 1 within the statistics' rounding)
    assert abs(a[0].sum().item() - 2 * chunk) <= 1e-6 * 2 * chunk
    b = _zeros(k, d)
    gmm.gmm_estep_accumulate_ring(x, n, *th, *b, chunk, ring, staging, ws, copy_stream=copy)
    c = _zeros(k, d)
    gmm.gmm_estep_accumulate(torch.from_numpy(x).cuda(), *th, *c, gmm.workspace(n, d, k))
    torch.cuda.synchronize()
    assert abs(b[0].sum().item() - n) <= 1e-6 * n
    assert abs(b[3].item() - c[3].item()) <= 1e-9 * abs(c[3].item())
