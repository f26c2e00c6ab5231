"""The out-of-core E-step: data in page-locked host memory, uploaded in chunks on a second
stream while the previous chunk's E-step runs.  Its statistics must equal, bit for bit, those
of gmm_estep_accumulate called chunk by chunk on device copies of the same rows, also across
EM iterations (the staging buffer is reused while earlier work may still read it), and match
the checker."""
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


@pytest.mark.parametrize("n,d,kt,k,chunk", [(50001, 128, 24, 64, 12000), (9000, 40, 6, 9, 9000),
                                            (20000, 300, 10, 30, 7001)])
def test_streamed_equals_chunk_by_chunk_calls(n, d, kt, k, chunk):
    import torch
    import paper_2606_10896_amd as gmm
    w = g.custom(f"stream{n}_{d}", n, d, kt, k, data_seed=5 + d, init_seed=6 + k)
    x, th0 = g.make(w)
    _say(f"  streamed E-step n={n} d={d} k={k} chunk={chunk}")
    xh = torch.from_numpy(x).pin_memory()
    rows = min(chunk, n)
    staging = torch.empty(2 * rows * d, dtype=torch.float32, device="cuda")
    ws = gmm.workspace(rows, d, k)
    copy = torch.cuda.Stream()
    chunks = [torch.from_numpy(x[r0:r0 + rows]).cuda() for r0 in range(0, n, rows)]
    ws_ref = gmm.workspace(rows, d, k)
    tha = [torch.from_numpy(a).cuda() for a in th0]
    thb = [torch.from_numpy(a).cuda() for a in th0]
    for it in range(3):
        a = _zeros(k, d)
        gmm.gmm_estep_accumulate_streamed(xh, *tha, *a, chunk, staging, ws, copy_stream=copy)
        b = _zeros(k, d)
        for xc in chunks:
            gmm.gmm_estep_accumulate(xc, *thb, *b, ws_ref)
        torch.cuda.synchronize()
        for u, v in zip(a, b):
            assert torch.equal(u, v), f"iteration {it}: streamed and chunked statistics differ"
        if it == 0:
            ref = oracle.estep(x, *th0)
            st = dict(nk=a[0].cpu().numpy(), s=a[1].cpu().numpy(), q=a[2].cpu().numpy(),
                      loglik=a[3].item())
            _say("  ", check_stats(st, ref, "streamed t=0"))
        gmm.gmm_mstep(*a[:3], float(n), *tha)
        gmm.gmm_mstep(*b[:3], float(n), *thb)
    torch.cuda.synchronize()
    for u, v in zip(tha, thb):
        assert torch.equal(u, v)


def test_concurrent_streamed_calls_on_two_streams():
    """Two out-of-core E-steps in flight at once, on two compute streams with their own copy
    streams, staging buffers and workspaces: each call orders its uploads with events of its
    own, so both results equal those of the same calls made one after the other."""
    import torch
    import paper_2606_10896_amd as gmm
    sets = []
    for i, (n, d, k, chunk) in enumerate([(30001, 64, 16, 7000), (24000, 64, 16, 5000)]):
        w = g.custom(f"conc{i}", n, d, 8, k, data_seed=40 + i, init_seed=50 + i)
        x, th = g.make(w)
        sets.append(dict(xh=torch.from_numpy(x).pin_memory(), th=[torch.from_numpy(a).cuda() for a in th],
                         chunk=chunk, k=k, d=d,
                         staging=torch.empty(2 * chunk * d, dtype=torch.float32, device="cuda"),
                         ws=gmm.workspace(chunk, d, k), copy=torch.cuda.Stream(),
                         stream=torch.cuda.Stream()))
    # one after the other
    seq = []
    for s in sets:
        out = _zeros(s["k"], s["d"])
        gmm.gmm_estep_accumulate_streamed(s["xh"], *s["th"], *out, s["chunk"], s["staging"], s["ws"],
                                          copy_stream=s["copy"])
        torch.cuda.synchronize()
        seq.append(out)
    # both in flight: each enqueued on its own stream before either is waited for
    par = [_zeros(s["k"], s["d"]) for s in sets]
    torch.cuda.synchronize()
    for s, out in zip(sets, par):
        gmm.gmm_estep_accumulate_streamed(s["xh"], *s["th"], *out, s["chunk"], s["staging"], s["ws"],
                                          stream=s["stream"], copy_stream=s["copy"])
    torch.cuda.synchronize()
    for i, (a, b) in enumerate(zip(seq, par)):
        for u, v in zip(a, b):
            assert torch.equal(u, v), f"set {i}: concurrent and sequential statistics differ"
    _say("  two concurrent streamed E-steps equal the sequential ones")
