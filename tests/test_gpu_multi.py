"""GPU parity of the multi-instance scheduling solution against the oracle, bit for bit:
instance assignment (sched_assign) on hand-worked and random cases, and every instance's
chains of sched_anneal_multi (start order, records, final and best orders) plus the
per-instance winners gathered by sched_multi_best."""
import json
import os
import sys

import numpy as np
import pytest

sys.path.insert(0, os.path.dirname(__file__))
from gpu_helpers import oracle_chains  # noqa: E402

from paper_2504_14966_amd.workloads import Model, Queue, multi_workload, random_queue  # noqa: E402

pytestmark = pytest.mark.gpu
GOLD = os.path.join(os.path.dirname(__file__), "golden", "worked_assignment.json")


@pytest.fixture(scope="module")
def sl():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2504_14966_amd.sloanneal as m
    m.load_library()
    return m


def _assign(sl, q, cap):
    import torch
    dq = sl.DeviceQueue.from_queue(q)
    out = sl.sched_assign(dq, torch.tensor(cap, dtype=torch.int64, device="cuda"))
    return out.cpu().numpy()


def test_assign_worked(sl):
    with open(GOLD) as f:
        g = json.load(f)
    for c in g["cases"]:
        need = c["need"]
        q = Queue(np.array([x - 1 for x in need], np.uint16), np.ones(len(need), np.uint16),
                  np.zeros(len(need), np.uint8), np.zeros(len(need), np.uint32))
        assert _assign(sl, q, c["capacity"]).tolist() == c["inst"], c["name"]


@pytest.mark.parametrize("seed", range(6))
def test_assign_random(sl, orc, seed):
    rng = np.random.default_rng(seed)
    I = [1, 2, 7, 33, 64, 5][seed]
    q = random_queue(rng, int(rng.integers(1, 1025)), max_in=4000, max_out=1000)
    cap = rng.integers(1000, 60000, size=I).astype(np.int64)
    assert np.array_equal(_assign(sl, q, cap), orc.assign(q, I, cap))


@pytest.mark.parametrize("seed", range(3))
def test_assign_wide_capacities(sl, orc, seed):
    # capacities from 2^25 tokens up take the 64-bit assignment; mixed with small ones too
    rng = np.random.default_rng(40 + seed)
    I = [3, 17, 64][seed]
    q = random_queue(rng, int(rng.integers(200, 1025)), max_in=60000, max_out=60000)
    cap = rng.integers(1 << 25, 1 << 26, size=I).astype(np.int64)
    cap[::2] = rng.integers(1000, 200000, size=len(cap[::2]))
    assert np.array_equal(_assign(sl, q, cap), orc.assign(q, I, cap))


def test_assign_narrow_edges(sl, orc):
    # capacities just below 2^25, requests of up to 2 * 65535 tokens, overdrawn instances
    rng = np.random.default_rng(7)
    q = random_queue(rng, 1024, max_in=65535, max_out=65535)
    for cap in ([(1 << 25) - 1] * 5, [1, 2, 3], [131070, 131069, 1], [1 << 20] * 64):
        cap = np.array(cap, np.int64)
        assert np.array_equal(_assign(sl, q, cap), orc.assign(q, len(cap), cap)), cap[:4]


def _check_instances(sl, orc, q, m, inst, I, C, iters, T0, alpha, seed, search, sample):
    import torch
    dq = sl.DeviceQueue.from_queue(q)
    inst_t = torch.tensor(inst, dtype=torch.int32, device="cuda")
    s_dev = sl.Search(*search) if search else None
    mws = sl.sched_anneal_multi(dq, m, inst_t, I, C, iters, T0, alpha, seed, search=s_dev)
    orders, keys, counts = sl.sched_multi_best(mws)
    torch.cuda.synchronize()
    orders, keys, counts = sl.as_u16(orders), keys.cpu().numpy(), counts.cpu().numpy()
    off = 0
    s_orc = orc.Search(*search) if search else None
    for k in range(I):
        sq, ids = orc.sub_queue(q, inst, k)
        assert counts[k] == sq.n
        if sq.n == 0:
            assert keys[k].tolist() == [-1, -1, -1]
            continue
        w = mws.instance(k)
        rec, cur, best = sl.sched_chains(w, sq.n, C, perms=True)
        st, info = sl.sched_start_info(w, sq.n)
        torch.cuda.synchronize()
        rec, cur, best = rec.cpu().numpy(), sl.as_u16(cur), sl.as_u16(best)
        oi = orc.start(sq, m, s_orc)
        assert sl.as_u16(st).tolist() == oi[0].tolist(), k
        assert info.cpu().numpy().tolist() == [oi[1], oi[3], oi[4], int(oi[2])], k
        # instance k's chain c is the single-queue chain with Philox chain index k * C + c
        want = oracle_chains(sq, m, [k * C + c for c in sample], iters, T0, alpha, seed, oi, search)
        for c in sample:
            wrec, wcur, wbest = want[k * C + c]
            assert rec[c].tolist() == wrec.tolist(), (k, c)
            assert cur[c].tolist() == wcur.tolist() and best[c].tolist() == wbest.tolist(), (k, c)
        win = max(range(C), key=lambda c: (rec[c, 2], -rec[c, 3], -c)) if not (search and search[0]) else None
        if win is not None:
            assert keys[k].tolist() == [rec[win, 2], rec[win, 3], win], k
        c = int(keys[k, 2])
        assert orders[off:off + sq.n].tolist() == ids[best[c]].tolist(), k
        off += sq.n
    assert sorted(orders.tolist()) == list(range(q.n))


@pytest.mark.parametrize("policy,search", [(0, None), (1, None), (0, (1, 5, 0)), (1, (0, 3, 1))])
def test_anneal_multi_random(sl, orc, policy, search):
    rng = np.random.default_rng(10 + policy)
    q = random_queue(rng, 150, max_in=1500, max_out=40, thr_hi=600_000)
    m = Model(6, policy, p0=2000, p1=40, d0=8000, d1=300, d2=2)
    inst = orc.assign(q, 5, [3000, 2500, 2000, 4000, 1000])
    _check_instances(sl, orc, q, m, inst, 5, 24, 400, 0.8, 0.99, 3, search, range(0, 24, 5))


def test_anneal_multi_empty_and_single_instances(sl, orc):
    rng = np.random.default_rng(4)
    q = random_queue(rng, 30, max_in=1500, max_out=40, thr_hi=600_000)
    m = Model(4, 0, p0=2000, p1=40, d0=8000, d1=300, d2=2)
    inst = np.zeros(q.n, np.int32)
    inst[::7] = 2                  # instance 1 has no request
    _check_instances(sl, orc, q, m, inst, 3, 8, 300, 1.0, 0.99, 1, None, range(8))
    _check_instances(sl, orc, q, m, np.zeros(q.n, np.int32), 1, 8, 300, 1.0, 0.99, 1, None, range(8))


def test_anneal_multi_one_request_instance(sl, orc):
    rng = np.random.default_rng(6)
    q = random_queue(rng, 40, max_in=1500, max_out=40, thr_hi=600_000)
    m = Model(8, 0, p0=2000, p1=40, d0=8000, d1=300, d2=2)
    inst = np.zeros(q.n, np.int32)
    inst[5] = 1                    # instance 1 serves a single request
    inst[20:] = 2
    _check_instances(sl, orc, q, m, inst, 3, 16, 300, 1.0, 0.99, 2, None, range(16))


@pytest.mark.parametrize("B,search", [(48, None), (48, (1, 4, 1)), (33, (0, 7, 0)), (64, None)])
def test_anneal_multi_batch_per_wave(sl, orc, B, search):
    # batches of more than 32 requests: the one-batch-per-wave delta kernel per instance
    rng = np.random.default_rng(20 + B)
    q = random_queue(rng, 300, max_in=1500, max_out=40, thr_hi=900_000)
    m = Model(B, 0, p0=2000, p1=40, d0=8000, d1=300, d2=2)
    inst = orc.assign(q, 3, [9000, 6000, 4000])
    _check_instances(sl, orc, q, m, inst, 3, 20, 300, 0.8, 0.99, 5, search, range(0, 20, 3))


def test_anneal_multi_static_wide(sl, orc):
    # 2 (d1 + d2 l_in) + d2 beyond 24 bits: static admission on the full-replay kernel
    rng = np.random.default_rng(31)
    q = random_queue(rng, 120, max_in=1500, max_out=40, thr_hi=2_000_000_000)
    assert int(q.in_len.max()) * 2 * 8000 > 1 << 24
    m = Model(8, 0, p0=2000, p1=40, d0=8000, d1=300, d2=8000)
    inst = orc.assign(q, 4, [20000, 15000, 9000, 6000])
    _check_instances(sl, orc, q, m, inst, 4, 12, 300, 1.0, 0.99, 7, None, range(0, 12, 4))


@pytest.mark.parametrize("B,search", [(1, None), (4, (1, 6, 0)), (16, None), (8, (1, 9, 1))])
def test_anneal_multi_small_instances(sl, orc, B, search):
    # every instance at most 64 requests: the register kernel per instance
    rng = np.random.default_rng(70 + B)
    q = random_queue(rng, 130, max_in=1500, max_out=40, thr_hi=900_000)
    m = Model(B, 0, p0=2000, p1=40, d0=8000, d1=300, d2=2)
    inst = orc.assign(q, 4, [3000, 3000, 3000, 3000])
    assert max(np.bincount(inst, minlength=4)) <= 64
    _check_instances(sl, orc, q, m, inst, 4, 10, 300, 0.8, 0.99, 6, search, range(0, 10, 3))


def test_anneal_multi_small_instances_wide_timeline(sl, orc):
    # register kernel per instance with the timeline above 2^32 (64-bit starts and sums)
    rng = np.random.default_rng(77)
    q = random_queue(rng, 100, max_in=3000, max_out=250, thr_hi=4_000_000_000)
    m = Model(16, 0, p0=5_000_000, p1=100, d0=16_000_000, d1=1000, d2=3)
    inst = (np.arange(q.n) % 3).astype(np.int32)
    _check_instances(sl, orc, q, m, inst, 3, 8, 200, 2.0, 0.99, 4, None, range(0, 8, 3))


def test_multi_workload_sampled(sl, orc):
    W = multi_workload()
    I, cap = W.extra["instances"], W.extra["capacity"]
    inst = _assign(sl, W.queue, cap)
    assert np.array_equal(inst, orc.assign(W.queue, I, cap))
    _check_instances(sl, orc, W.queue, W.model, inst, I, W.chains, 400, W.T0, W.alpha, W.seed, None, (0, 511))


@pytest.mark.parametrize("seed", range(12))
def test_anneal_multi_random_sweep(sl, orc, seed):
    # random instance counts and capacities: instances of one to three positions per lane
    # (up to 192 requests), or the delta kernels above, in one launch; both objectives
    rng = np.random.default_rng(8000 + seed)
    I = int(rng.integers(1, 7))
    n = int(rng.integers(I, 500))
    B = int(rng.choice([1, 2, 4, 8, 16, 16, 16, 24]))
    q = random_queue(rng, n, max_in=1500, max_out=60, thr_hi=900_000)
    m = Model(B, 0, p0=2000, p1=40, d0=8000, d1=300, d2=2)
    caps = [int(x) for x in rng.integers(2000, 60000, I)]
    inst = orc.assign(q, I, caps)
    search = None if rng.random() < 0.5 else (1, int(rng.integers(1, 20)), int(rng.integers(0, 2)))
    _check_instances(sl, orc, q, m, inst, I, 6, 150, 0.8, 0.99, seed, search, range(0, 6, 2))
