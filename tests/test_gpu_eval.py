"""GPU parity of sched_eval and sched_gen_perms against the CPU oracle (bit-exact).

Cases: the hand-worked timelines; all 40320 orders of the 8-request workload; random
queues across batch sizes (powers of two and not), both admission policies, ragged last
batches and per-request detail; rows that are not permutations; the 128-request
evaluation workload at its full 2^20 rows, every row checked against the oracle.
"""
import hashlib
import json
import os
import sys
from itertools import permutations

import numpy as np
import pytest

sys.path.insert(0, os.path.dirname(__file__))
from gpu_helpers import oracle_fy_rows, oracle_rows  # noqa: E402

from paper_2504_14966_amd.workloads import Model, Queue, random_queue, workload  # noqa: E402

pytestmark = pytest.mark.gpu
GOLD = os.path.join(os.path.dirname(__file__), "golden", "worked_timelines.json")


@pytest.fixture(scope="module")
def sl():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2504_14966_amd.sloanneal as m
    m.load_library()
    return m


def _eval(sl, q, m, perms, detail=False):
    dq = sl.DeviceQueue.from_queue(q)
    r = sl.sched_eval(dq, m, sl.perms_to_device(perms), detail=detail)
    if detail:
        return r[0].cpu().numpy(), r[1].cpu().numpy()
    return r.cpu().numpy()


def test_worked_timelines(sl, orc):
    g = json.load(open(GOLD))
    qd = g["queue"]
    q = Queue(np.array(qd["in_len"], np.uint16), np.array(qd["out_len"], np.uint16), np.array(qd["kind"], np.uint8),
              np.array(qd["thr_us"], np.uint32))
    for case in g["cases"]:
        m = Model(case["max_batch"], case["policy"], **g["model"])
        out, det = _eval(sl, q, m, np.array([case["perm"]]), detail=True)
        assert out[0].tolist() == [case["n"], case["t"]], case["name"]
        assert det[0, :, 0].tolist() == case["ttft"] and det[0, :, 1].tolist() == case["e2e"], case["name"]
    for table, B, pol in (("static_b2", 2, 0), ("continuous_b2", 2, 1), ("b1", 1, 0), ("b1", 1, 1)):
        m = Model(B, pol, **g["model"])
        keys = list(g["all_orders"][table].keys())
        perms = np.array([[int(x) for x in k.split(",")] for k in keys])
        out = _eval(sl, q, m, perms)
        assert [list(v) for v in out.tolist()] == [g["all_orders"][table][k] for k in keys]


def test_all_orders_of_workload_1(sl, orc):
    W = workload(1)
    perms = np.array(list(permutations(range(8))), dtype=np.uint16)
    got = _eval(sl, W.queue, W.model, perms)
    want = oracle_rows(W.queue, W.model, perms)
    assert np.array_equal(got, want)
    bn, bt, bp, cnt = orc.brute(W.queue, W.model)
    best = max(range(len(got)), key=lambda r: (got[r, 0], -got[r, 1], -r))
    assert (got[best, 0], got[best, 1]) == (bn, bt) and perms[best].tolist() == bp.tolist()
    assert int(((got[:, 0] == bn) & (got[:, 1] == bt)).sum()) == cnt


@pytest.mark.parametrize("n,B,policy", [(1, 1, 0), (1, 4, 1), (2, 1, 1), (5, 2, 0), (7, 3, 0), (7, 3, 1), (13, 5, 0),
                                        (13, 5, 1), (33, 8, 0), (64, 64, 0), (65, 64, 1), (100, 7, 1),
                                        (100, 33, 0), (130, 17, 1), (257, 64, 0), (300, 1, 0), (300, 2, 1),
                                        (1024, 64, 0), (1024, 64, 1), (1024, 48, 0), (512, 31, 1)])
def test_random_queues_with_detail(sl, orc, n, B, policy):
    rng = np.random.default_rng(1000 * n + 10 * B + policy)
    q = random_queue(rng, n, max_in=int(rng.choice([64, 2048, 65535])), max_out=int(rng.choice([8, 200, 1024])))
    m = Model(B, policy, p0=int(rng.integers(0, 3000)), p1=int(rng.integers(0, 50)), d0=int(rng.integers(0, 9000)),
              d1=int(rng.integers(0, 400)), d2=int(rng.integers(0, 3)))
    rows = 6 if n >= 512 else 24
    perms = np.stack([rng.permutation(n) for _ in range(rows)]).astype(np.uint16)
    out, det = _eval(sl, q, m, perms, detail=True)
    for r in range(rows):
        nn, tt, ttft, e2e = orc.replay(q, m, perms[r], detail=True)
        assert out[r].tolist() == [nn, tt], (r, n, B, policy)
        assert np.array_equal(det[r, :, 0], ttft) and np.array_equal(det[r, :, 1], e2e), (r, n, B, policy)


def _timeline_end(q, m):
    # the end of the timeline of any order under static batches
    li, lo = q.in_len.astype(object), q.out_len.astype(object)
    return sum(m.p0 + m.p1 * li) + (m.d0 + m.d1) * sum(lo) + m.d2 * sum(lo * li + lo * (lo + 1) // 2)


@pytest.mark.parametrize("n,B,wide", [(1, 1, False), (7, 3, False), (33, 8, False), (64, 64, False),
                                      (100, 33, False), (257, 64, False), (300, 1, False), (1024, 64, False),
                                      (1024, 48, False), (200, 20, False), (90, 32, False), (50, 2, False),
                                      (64, 16, True), (130, 17, True), (64, 1, True), (200, 5, True)])
def test_static_rows_without_detail(sl, orc, n, B, wide):
    # totals only: a timeline within 32 bits takes the 32-bit start scan and latency sum,
    # a wider one the 64-bit path
    rng = np.random.default_rng(77 * n + B)
    if wide:
        q = random_queue(rng, n, max_in=3000, max_out=250, thr_hi=4_000_000_000)
        m = Model(B, 0, p0=5_000_000, p1=100, d0=16_000_000 // max(1, B // 16), d1=1000, d2=3)
    else:
        q = random_queue(rng, n, max_in=2048, max_out=200)
        m = Model(B, 0, p0=2000, p1=40, d0=8000, d1=300, d2=2)
    assert (_timeline_end(q, m) >= 2**32 - 2) == wide
    rows = 8 if n >= 512 else 24
    perms = np.stack([rng.permutation(n) for _ in range(rows)]).astype(np.uint16)
    out = _eval(sl, q, m, perms)
    for r in range(rows):
        nn, tt = orc.replay(q, m, perms[r])[:2]
        assert out[r].tolist() == [nn, tt], (r, n, B)


def test_non_permutation_rows(sl, orc):
    W = workload(2)
    n = W.queue.n
    rng = np.random.default_rng(3)
    perms = np.stack([rng.permutation(n) for _ in range(8)]).astype(np.uint16)
    perms[1, 5] = perms[1, 6]           # duplicate
    perms[3, 0] = n                     # out of range
    perms[5, :] = 0                     # all equal
    perms[6, 63] = 0xFFFF
    out = _eval(sl, W.queue, W.model, perms)
    for r in range(8):
        want = orc.replay(W.queue, W.model, perms[r])
        assert out[r].tolist() == list(want)
    assert out[1].tolist() == [-1, -1] and out[3].tolist() == [-1, -1] and out[5].tolist() == [-1, -1]


def test_empty_batch_of_rows(sl):
    import torch
    W = workload(1)
    dq = sl.DeviceQueue.from_queue(W.queue)
    out = sl.sched_eval(dq, W.model, torch.empty((0, 8), dtype=torch.int16, device="cuda"))
    assert out.shape == (0, 2)


def test_bad_queue_entries_rejected(sl):
    # the queue's contents are checked on the device: every row reads (-2, code), detail
    # is left untouched; both admission policies, with and without detail
    import torch
    W = workload(1)
    perms = np.stack([np.arange(8, dtype=np.uint16), np.arange(8, dtype=np.uint16)[::-1]])
    for policy in (0, 1):
        m = Model(4, policy, p0=2000, p1=40, d0=8000, d1=300, d2=2)
        for field, val in (("out_len", 0), ("kind", 3), ("thr_us", 0xFFFFFFFF)):
            q = Queue(W.queue.in_len.copy(), W.queue.out_len.copy(), W.queue.kind.copy(), W.queue.thr_us.copy())
            getattr(q, field)[2] = val
            assert _eval(sl, q, m, perms).tolist() == [[-2, sl.SCHED_EINVAL]] * 2
            dq = sl.DeviceQueue.from_queue(q)
            det = torch.full((2, 8, 2), 7, dtype=torch.int64, device="cuda")
            out, _ = sl.sched_eval(dq, m, sl.perms_to_device(perms), detail=det)
            assert out.cpu().tolist() == [[-2, sl.SCHED_EINVAL]] * 2
            assert bool((det == 7).all())
        big = Model(4, policy, p0=2000, p1=40, d0=2**55, d1=300, d2=2)
        assert _eval(sl, W.queue, big, perms).tolist() == [[-2, sl.SCHED_ERANGE]] * 2
    # the layout evaluation checks the same way
    q = Queue(W.queue.in_len.copy(), W.queue.out_len.copy(), W.queue.kind.copy(), W.queue.thr_us.copy())
    q.out_len[5] = 0
    st = np.zeros((2, 8), np.uint8)
    st[:, ::4] = 1
    out = sl.sched_eval_batches(sl.DeviceQueue.from_queue(q), W.model, sl.perms_to_device(perms),
                                sl.starts_to_device(st))
    assert out.cpu().tolist() == [[-2, sl.SCHED_EINVAL]] * 2


def test_fisher_yates_family(sl, orc):
    got = sl.as_u16(sl.sched_gen_perms(0, 128, 4096, row0=1000))
    for r in list(range(0, 4096, 97)) + [4095]:
        assert got[r].tolist() == orc.fy_perm(0, 128, 1000 + r).tolist()
    got = sl.as_u16(sl.sched_gen_perms(2**40 + 7, 1024, 64))
    for r in (0, 31, 63):
        assert got[r].tolist() == orc.fy_perm(2**40 + 7, 1024, r).tolist()
    got = sl.as_u16(sl.sched_gen_perms(5, 1, 3))
    assert got.tolist() == [[0], [0], [0]]


def test_eval_workload_every_row(sl, orc):
    """Workload 5: all 2^20 Fisher-Yates orders of 128 requests, in the benchmark's launch
    shape. The oracle regenerates every order from its own Philox and scores it (in worker
    processes); the GPU's orders must hash equal block by block and every (n, t) must agree."""
    import torch
    W = workload(5)
    dq = sl.DeviceQueue.from_queue(W.queue)
    perms = sl.sched_gen_perms(W.perm_seed, W.queue.n, W.eval_rows)
    out = sl.sched_eval(dq, W.model, perms)
    out2 = sl.sched_eval(dq, W.model, perms)
    torch.cuda.synchronize()
    assert torch.equal(out, out2)
    o = out.cpu().numpy()
    host = sl.as_u16(perms)
    blocks = oracle_fy_rows(W.queue, W.model, W.perm_seed, W.eval_rows)
    for lo, hi, digest, want in blocks:
        assert hashlib.sha256(np.ascontiguousarray(host[lo:hi]).tobytes()).hexdigest() == digest, (lo, hi)
        bad = np.flatnonzero((o[lo:hi] != want).any(axis=1))
        assert bad.size == 0, (lo + bad[:5]).tolist()
    assert sum(hi - lo for lo, hi, _, _ in blocks) == W.eval_rows
    assert (o[:, 0] >= 0).all() and (o[:, 0] <= 128).all() and (o[:, 1] > 0).all()
