"""The C ABI from several host threads at once.

Every entry point is documented as thread-safe, and the library owns one
shared structure, the route-plan cache (built on first use of a (device, n,
B, L), on a private stream, under a lock).  Here four host threads, each on
its own HIP stream, call the forward and the backward for lengths whose plans
do not exist yet, so that first builds, cache hits and kernel launches
interleave; every result must equal, bitwise, the same call made alone on one
thread.  (ctypes releases the interpreter lock around each library call, so
the calls do run concurrently.)
"""

import threading

import pytest
import torch

import paper_2608_20427_amd as bf1
from paper_2608_20427_amd import synth

pytestmark = pytest.mark.gpu

LENGTHS = [517, 1100, 2049, 3000, 777, 1500, 64 * 9, 2500]


@pytest.fixture(scope="module", autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    bf1.load()
    yield
    torch.cuda.synchronize()


def _inputs(n):
    w = synth.Workload("thr", 1, n, 4, 2, 128, 64, 2, seed=40 + n)
    q, k, v = synth.make_qkv(w, device="cuda")
    do = synth.make_grad_out(w, device="cuda")
    return w, q, k, v, do


def _run(w, q, k, v, do):
    o, lse = bf1.attn_fwd(q, k, v, B=w.b, L=w.L)
    dq, dk, dv = bf1.attn_bwd(q, k, v, o, do, lse, w.b, w.L)
    return o, lse, dq, dk, dv


def test_concurrent_calls_match_single_thread():
    cases = [_inputs(n) for n in LENGTHS]
    torch.cuda.synchronize()
    # reference: one thread, plans built one at a time
    bf1.release_plans()
    ref = []
    for c in cases:
        r = _run(*c)
        torch.cuda.synchronize()
        ref.append([t.clone() for t in r])
    # four threads, fresh plan cache: every length's first build races with
    # the other threads' builds and launches
    bf1.release_plans()
    got = [None] * len(cases)
    errors = []

    def worker(tid):
        try:
            s = torch.cuda.Stream()
            with torch.cuda.stream(s):
                for rep in range(2):
                    for i in range(tid, len(cases), 4):
                        r = _run(*cases[i])
                        s.synchronize()
                        if rep == 1:
                            got[i] = [t.clone() for t in r]
        except Exception as e:  # reported below, on the main thread
            errors.append((tid, repr(e)))

    threads = [threading.Thread(target=worker, args=(t,)) for t in range(4)]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=240)
    torch.cuda.synchronize()
    assert not any(t.is_alive() for t in threads), "a worker thread did not finish"
    assert not errors, errors
    for i, n in enumerate(LENGTHS):
        for name, a, b in zip(("O", "LSE", "dQ", "dK", "dV"), got[i], ref[i]):
            same = torch.equal(a.view(torch.int16), b.view(torch.int16)) if a.dtype == torch.bfloat16 \
                else torch.equal(a, b)
            assert same, (n, name)
