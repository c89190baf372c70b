"""sched_anneal_noalloc (annealing in the library's fixed device scratch, for callers that
cannot allocate) against sched_anneal + sched_best on a caller's workspace: the same best
order and key, bit for bit, on two calls in a row, the second with a smaller input; sizes
beyond the scratch are refused before anything runs."""
import ctypes as C

import numpy as np
import pytest

from paper_2504_14966_amd.workloads import Model, random_queue, workload

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sl():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2504_14966_amd.sloanneal as m
    m.load_library()
    return m


def _with_ws(sl, dq, m, chains, iters, T0, alpha, seed):
    ws = sl.sched_anneal(dq, m, chains, iters, T0, alpha, seed)
    return sl.sched_best(ws, dq.n)


def _case(sl, q, m, chains, iters, T0, alpha, seed):
    import torch
    dq = sl.DeviceQueue.from_queue(q)
    perm, key = sl.sched_anneal_noalloc(dq, m, chains, iters, T0, alpha, seed)
    wperm, wkey = _with_ws(sl, dq, m, chains, iters, T0, alpha, seed)
    torch.cuda.synchronize()
    assert key.cpu().tolist() == wkey.cpu().tolist()
    assert sl.as_u16(perm).tolist() == sl.as_u16(wperm).tolist()
    assert sorted(sl.as_u16(perm).tolist()) == list(range(q.n))
    return key.cpu().tolist()


def test_noalloc_matches_workspace_call_twice(sl):
    # first call at the burst workload's full size (1024 requests, 4096 chains), then a
    # smaller queue in the same scratch
    W = workload(4)
    k1 = _case(sl, W.queue, W.model, W.chains, 300, W.T0, W.alpha, W.seed)
    assert k1[0] > 0
    rng = np.random.default_rng(17)
    q = random_queue(rng, 40, max_in=2000, max_out=60, thr_hi=2_000_000)
    m = Model(8, 0, p0=2000, p1=40, d0=8000, d1=300, d2=2)
    _case(sl, q, m, 96, 800, 1.0, 0.995, 5)


def test_noalloc_other_policies(sl):
    rng = np.random.default_rng(3)
    q = random_queue(rng, 150, max_in=2000, max_out=60, thr_hi=5_000_000)
    for policy, B in ((1, 12), (2, 8), (0, 64)):
        _case(sl, q, Model(B, policy, p0=2000, p1=40, d0=8000, d1=300, d2=2), 200, 400, 1.0, 0.99, 11)


def test_noalloc_refuses_sizes_beyond_the_scratch(sl):
    L = sl.load_library()
    W = workload(4)
    dq = sl.DeviceQueue.from_queue(W.queue)
    q, m = dq.c(), sl._model(W.model)
    limit = 32 << 20
    assert sl.ws_bytes(1024, 5404) <= limit < sl.ws_bytes(1024, 5405)
    rc = L.sched_anneal_noalloc(C.byref(q), C.byref(m), 5405, 10, 1.0, 0.9, 0, 256, 256, None)
    assert rc == sl.SCHED_ENOSPC
    assert b"SCHED_NOALLOC_MAX_BYTES" in L.sched_strerror(rc)
