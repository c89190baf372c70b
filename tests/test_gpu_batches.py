"""GPU parity of the joint search over order and batch sizes against the CPU oracle, bit
for bit: sched_eval_batches on random and adversarial (order, layout) rows, and
sched_anneal with SCHED_STATIC_SEARCH per chain (final and best orders and layouts, keys,
best iteration, accept count, trajectory digest) plus the cross-chain winner."""
import os
import sys

import numpy as np
import pytest

sys.path.insert(0, os.path.dirname(__file__))
from gpu_helpers import oracle_chains_batches, oracle_rows_batches  # noqa: E402

from paper_2504_14966_amd.workloads import (Model, Queue, random_layouts, random_queue,  # noqa: E402
                                            search_workload, workload)

pytestmark = pytest.mark.gpu
SEARCH = 2


@pytest.fixture(scope="module")
def sl():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2504_14966_amd.sloanneal as m
    m.load_library()
    return m


def _eval(sl, q, m, perms, starts, detail=False):
    import torch
    dq = sl.DeviceQueue.from_queue(q)
    res = sl.sched_eval_batches(dq, m, sl.perms_to_device(perms), sl.starts_to_device(starts), detail=detail)
    torch.cuda.synchronize()
    if detail:
        return res[0].cpu().numpy(), res[1].cpu().numpy()
    return res.cpu().numpy()


@pytest.mark.parametrize("wl,k", [(1, 512), (2, 2048), (5, 2048), (4, 256)])
def test_eval_batches_random_layouts(sl, orc, wl, k):
    W = workload(wl)
    q, B = W.queue, W.model.max_batch
    m = Model(B, SEARCH, W.model.p0, W.model.p1, W.model.d0, W.model.d1, W.model.d2)
    rng = np.random.default_rng(100 + wl)
    perms = np.stack([rng.permutation(q.n) for _ in range(k)]).astype(np.uint16)
    starts = random_layouts(rng, k, q.n, B)
    got = _eval(sl, q, m, perms, starts)
    want = oracle_rows_batches(q, m, perms, starts)
    assert np.array_equal(got, want)
    # the maximum-size layout through sched_eval_batches is sched_eval
    mx = np.stack([orc.max_starts(q.n, B)] * 64)
    import torch
    dq = sl.DeviceQueue.from_queue(q)
    plain = sl.sched_eval(dq, W.model, sl.perms_to_device(perms[:64])).cpu().numpy()
    assert np.array_equal(_eval(sl, q, m, perms[:64], mx), plain)
    torch.cuda.synchronize()


def test_eval_batches_detail_and_invalid_rows(sl, orc):
    W = workload(2)
    q, B = W.queue, W.model.max_batch
    m = Model(B, SEARCH, W.model.p0, W.model.p1, W.model.d0, W.model.d1, W.model.d2)
    rng = np.random.default_rng(7)
    k = 40
    perms = np.stack([rng.permutation(q.n) for _ in range(k)]).astype(np.uint16)
    starts = random_layouts(rng, k, q.n, B)
    starts[1, 0] = 0                      # no batch at position 0
    starts[2, :] = 0
    starts[2, 0] = 1                      # one batch of 64 > 16
    starts[3, 5] = 2                      # a flag that is not 0 or 1
    starts[4, :] = 0
    starts[4, ::16] = 1
    starts[4, 0] = 1                      # exactly 16 per batch: valid
    starts[5, :] = 0
    starts[5, ::17] = 1                   # 17 > 16: invalid
    perms[6, 3] = perms[6, 4]             # not a permutation
    perms[7, 0] = q.n                     # id out of range
    starts[8, :] = 1                      # all batches of one: valid
    out, det = _eval(sl, q, m, perms, starts, detail=True)
    for r in range(k):
        n_, t_, ttft, e2e = orc.replay_batches(q, m, perms[r], starts[r], detail=True)
        assert out[r].tolist() == [n_, t_], r
        if n_ >= 0:
            assert det[r, :, 0].tolist() == ttft.tolist() and det[r, :, 1].tolist() == e2e.tolist(), r
        else:
            assert not det[r].any(), r
    assert [out[r, 0] for r in (1, 2, 3, 5, 6, 7)] == [-1] * 6 and out[4, 0] >= 0 and out[8, 0] >= 0


@pytest.mark.parametrize("n,B,seed", [(1, 4, 0), (2, 1, 1), (3, 2, 2), (37, 5, 3), (64, 64, 4), (130, 33, 5),
                                      (1024, 64, 6), (1000, 7, 7)])
def test_eval_batches_edge_shapes(sl, orc, n, B, seed):
    rng = np.random.default_rng(seed)
    q = random_queue(rng, n, max_in=3000, max_out=200)
    m = Model(B, SEARCH, 2000, 40, 8000, 300, 2)
    k = 24
    perms = np.stack([rng.permutation(n) for _ in range(k)]).astype(np.uint16)
    starts = random_layouts(rng, k, n, B)
    starts[0] = 1
    starts[1] = orc.max_starts(n, B)
    assert np.array_equal(_eval(sl, q, m, perms, starts), orc.eval_rows_batches(q, m, perms, starts))


def _anneal(sl, q, m, chains, iters, T0, alpha, seed):
    import torch
    dq = sl.DeviceQueue.from_queue(q)
    ws = sl.sched_anneal(dq, m, chains, iters, T0, alpha, seed)
    rec, cur, best = sl.sched_chains(ws, q.n, chains, perms=True)
    cs, bs, ws_win = sl.sched_starts(ws, q.n, chains)
    bp, key = sl.sched_best(ws, q.n)
    torch.cuda.synchronize()
    return dict(rec=rec.cpu().numpy(), cur=sl.as_u16(cur), best=sl.as_u16(best), cur_starts=cs.cpu().numpy(),
                best_starts=bs.cpu().numpy(), win_starts=ws_win.cpu().numpy(), best_perm=sl.as_u16(bp),
                key=key.cpu().numpy())


def _check_chains(orc, res, q, m, sample, iters, T0, alpha, seed):
    info = orc.start(q, m)
    want = oracle_chains_batches(q, m, sample, iters, T0, alpha, seed, info)
    for c in sample:
        w = want[c]
        assert res["rec"][c].tolist() == w["rec"].tolist(), f"chain {c}"
        for f in ("cur", "best", "cur_starts", "best_starts"):
            assert res[f][c].tolist() == w[f].tolist(), f"chain {c} {f}"
    r = res["rec"]
    k = max(range(len(r)), key=lambda c: (r[c, 2], -r[c, 3], -c))
    assert res["key"].tolist() == [r[k, 2], r[k, 3], k]
    assert res["best_perm"].tolist() == res["best"][k].tolist()
    assert res["win_starts"].tolist() == res["best_starts"][k].tolist()
    for c in list(sample)[:4]:
        assert orc.replay_batches(q, m, res["cur"][c], res["cur_starts"][c]) == (r[c, 0], r[c, 1])
        assert orc.replay_batches(q, m, res["best"][c], res["best_starts"][c]) == (r[c, 2], r[c, 3])


def test_anneal_search_worked_queue(sl, orc):
    """The 3-request queue whose joint optimum needs a batch of one (hand-worked: (3, 132036))."""
    q = Queue(np.array([100, 50, 200], np.uint16), np.array([2, 3, 1], np.uint16), np.array([0, 2, 1], np.uint8),
              np.array([8000, 70000, 9200], np.uint32))
    m = Model(2, SEARCH, 2000, 40, 8000, 300, 2)
    res = _anneal(sl, q, m, 64, 300, 1.0, 0.99, 0)
    _check_chains(orc, res, q, m, range(64), 300, 1.0, 0.99, 0)
    assert res["key"][:2].tolist() == [3, 132036]


@pytest.mark.parametrize("n,B,chains,iters,seed", [(1, 3, 5, 40, 0), (2, 1, 8, 100, 1), (9, 4, 70, 700, 2),
                                                   (40, 7, 33, 900, 3), (100, 33, 20, 600, 4),
                                                   (64, 64, 10, 500, 5), (200, 17, 12, 500, 6),
                                                   (450, 40, 8, 400, 7), (1000, 64, 4, 300, 8),
                                                   (77, 3, 6, 600, 9), (130, 2, 6, 600, 10), (260, 5, 4, 500, 11)])
def test_anneal_search_random_queues(sl, orc, n, B, chains, iters, seed):
    rng = np.random.default_rng(seed)
    q = random_queue(rng, n, max_in=1500, max_out=40, thr_hi=400_000 * max(1, n // B))
    m = Model(B, SEARCH, 2000, 40, 8000, 300, 2)
    res = _anneal(sl, q, m, chains, iters, 1.0, 0.995, 11 + seed)
    _check_chains(orc, res, q, m, range(chains), iters, 1.0, 0.995, 11 + seed)


@pytest.mark.parametrize("wl,chains,iters,sample", [(1, 64, 2000, range(8)), (2, 1024, 2000, (0, 511, 1023)),
                                                     (4, 256, 300, (0, 255))])
def test_anneal_search_workloads(sl, orc, wl, chains, iters, sample):
    W = search_workload(wl)
    res = _anneal(sl, W.queue, W.model, chains, iters, W.T0, W.alpha, W.seed)
    _check_chains(orc, res, W.queue, W.model, sample, iters, W.T0, W.alpha, W.seed)


def test_starts_after_fixed_policy_runs(sl):
    W = workload(1)
    import torch
    dq = sl.DeviceQueue.from_queue(W.queue)
    ws = sl.sched_anneal(dq, W.model, 4, 50, W.T0, W.alpha, 0)
    cs, bs, win = sl.sched_starts(ws, W.queue.n, 4)
    torch.cuda.synchronize()
    want = [int(p % W.model.max_batch == 0) for p in range(W.queue.n)]
    assert all(row.tolist() == want for row in cs.cpu().numpy())
    assert all(row.tolist() == want for row in bs.cpu().numpy())
    assert win.cpu().numpy().tolist() == want


def _pq(rng, n, in_lo, in_hi, out_lo, out_hi, thr_hi):
    return Queue(rng.integers(in_lo, in_hi + 1, n).astype(np.uint16), rng.integers(out_lo, out_hi + 1, n).astype(np.uint16),
                 rng.integers(0, 3, n).astype(np.uint8), rng.integers(0, thr_hi, n).astype(np.uint32))


# Each case falls on one kernel path of the batch-size search: the delta kernel (32-bit
# offsets and timeline) or the full-replay kernel (64-bit everything).
SEARCH_PATHS = {
    # delta kernel: batch size 1 (squeeze and delay never allowed)
    "delta_b1": (lambda r: _pq(r, 300, 16, 2048, 1, 6, 4_000_000_000), Model(1, SEARCH, 2000, 40, 8000, 300, 2), 6, 300),
    # one batch of everything at the start (50 requests: the register search kernel); delays
    # open new last batches
    "delta_one_batch": (lambda r: _pq(r, 50, 16, 2048, 1, 300, 3_000_000), Model(64, SEARCH, 2000, 40, 8000, 300, 2), 8, 600),
    # delta kernel: equal output lengths (ties in every batch)
    "delta_ties": (lambda r: _pq(r, 90, 16, 64, 7, 7, 2_000_000), Model(12, SEARCH, 2000, 40, 8000, 300, 2), 8, 800),
    # full replay: pair costs beyond 24 bits
    "replay_wide": (lambda r: _pq(r, 48, 16, 2048, 8, 300, 4_000_000_000), Model(8, SEARCH, 2000, 40, 8000, 300, 1 << 22), 8, 300),
    # full replay: 32-bit offsets but a timeline longer than 2^32 us
    "replay_long_timeline": (lambda r: _pq(r, 200, 16, 2048, 5000, 20000, 4_000_000_000),
                             Model(2, SEARCH, 2000, 40, 8000, 300, 2), 4, 100),
}


@pytest.mark.parametrize("name", sorted(SEARCH_PATHS))
def test_anneal_search_paths(sl, orc, name):
    import zlib
    mk, m, chains, iters = SEARCH_PATHS[name]
    rng = np.random.default_rng(zlib.crc32(name.encode()))
    q = mk(rng)
    res = _anneal(sl, q, m, chains, iters, 0.7, 0.99, 5)
    _check_chains(orc, res, q, m, range(chains), iters, 0.7, 0.99, 5)


def test_batches_huge_times_one_batch_replay(sl, orc):
    # times from 2^57 on: the windowed replay's keys would not hold them, so sched_eval_batches
    # and the full-replay search chains take one batch per step (the timeline bound
    # 2^57 <= clock, and clock * n * (n + 2) < 2^62 keeps the range check)
    rng = np.random.default_rng(77)
    n, B = 3, 2
    q = random_queue(rng, n, max_in=1000, max_out=20, thr_hi=2**32 - 2)
    m = Model(B, SEARCH, 1 << 56, 3, 5, 7, 1)
    k = 24
    perms = np.stack([rng.permutation(n) for _ in range(k)]).astype(np.uint16)
    starts = random_layouts(rng, k, n, B)
    assert np.array_equal(_eval(sl, q, m, perms, starts), oracle_rows_batches(q, m, perms, starts))
    res = _anneal(sl, q, m, 4, 60, 0.7, 0.99, 9)
    _check_chains(orc, res, q, m, range(4), 60, 0.7, 0.99, 9)


@pytest.mark.parametrize("n,B", [(40, 6), (300, 16)])
def test_eval_batches_wide_model(sl, orc, n, B):
    # pair costs beyond 24 bits (d2 large): the windowed replay in 64-bit arithmetic
    rng = np.random.default_rng(n + B)
    q = random_queue(rng, n, max_in=3000, max_out=200, thr_hi=4_000_000_000)
    assert int(q.in_len.max()) * 2 * 9000 > 1 << 24
    m = Model(B, SEARCH, 2000, 40, 8000, 300, 9000)
    k = 48
    perms = np.stack([rng.permutation(n) for _ in range(k)]).astype(np.uint16)
    starts = random_layouts(rng, k, n, B)
    assert np.array_equal(_eval(sl, q, m, perms, starts), oracle_rows_batches(q, m, perms, starts))


@pytest.mark.parametrize("n,B", [(64, 16), (200, 5), (130, 17)])
def test_eval_batches_wide_timeline(sl, orc, n, B):
    # narrow pair costs but the timeline above 2^32: the windowed replay in 64 bits (below
    # 2^32 the 32-bit windows take over)
    rng = np.random.default_rng(3 * n + B)
    q = random_queue(rng, n, max_in=3000, max_out=250, thr_hi=4_000_000_000)
    m = Model(B, SEARCH, p0=5_000_000, p1=100, d0=16_000_000 // max(1, B // 16), d1=1000, d2=3)
    li, lo = q.in_len.astype(object), q.out_len.astype(object)
    assert sum(m.p0 + m.p1 * li) + (m.d0 + m.d1) * sum(lo) + m.d2 * sum(lo * li + lo * (lo + 1) // 2) > 2**32
    k = 32
    perms = np.stack([rng.permutation(n) for _ in range(k)]).astype(np.uint16)
    starts = random_layouts(rng, k, n, B)
    starts[0] = orc.max_starts(n, B)
    assert np.array_equal(_eval(sl, q, m, perms, starts), orc.eval_rows_batches(q, m, perms, starts))


@pytest.mark.parametrize("seed", range(12))
def test_eval_random_sweep(sl, orc, seed):
    # both evaluation calls over random shapes and the three width regimes: narrow timeline,
    # narrow pair costs with a timeline above 2^32, and 64-bit pair costs
    rng = np.random.default_rng(7000 + seed)
    regime = int(rng.integers(0, 3))
    n = int(rng.integers(1, 1025 if regime < 2 else 201))
    B = int(rng.integers(1, 65))
    if regime == 0:
        q = random_queue(rng, n, max_in=3000, max_out=200)
        kw = dict(p0=2000, p1=40, d0=8000, d1=300, d2=2)
    elif regime == 1:
        q = random_queue(rng, n, max_in=3000, max_out=250, thr_hi=4_000_000_000)
        kw = dict(p0=5_000_000, p1=100, d0=16_000_000 // max(1, min(n, B) // 16 + 1), d1=1000, d2=3)
    else:
        q = random_queue(rng, n, max_in=3000, max_out=200, thr_hi=4_000_000_000)
        kw = dict(p0=2000, p1=40, d0=8000, d1=300, d2=9000)
    # the library's int64 bound (every prefill, then per decode step a full batch of the
    # longest contexts; the sum over requests and the objective's scale below 2^62)
    b = min(n, B)
    step = kw["d0"] + kw["d1"] * b + kw["d2"] * b * (int(q.in_len.max()) + int(q.out_len.max()))
    clock = sum(kw["p0"] + kw["p1"] * int(x) for x in q.in_len) + int(q.out_len.astype(np.int64).sum()) * step
    assert clock * n * (n + 2) < 2**62
    k = 8 if n > 256 else 16
    perms = np.stack([rng.permutation(n) for _ in range(k)]).astype(np.uint16)
    # fixed batches through sched_eval
    m0 = Model(B, 0, **kw)
    dq = sl.DeviceQueue.from_queue(q)
    out = sl.sched_eval(dq, m0, sl.perms_to_device(perms)).cpu().numpy()
    for r in range(k):
        assert out[r].tolist() == list(orc.replay(q, m0, perms[r])[:2]), (r, n, B, regime)
    # explicit layouts through sched_eval_batches
    m2 = Model(B, SEARCH, **kw)
    starts = random_layouts(rng, k, n, B)
    assert np.array_equal(_eval(sl, q, m2, perms, starts), orc.eval_rows_batches(q, m2, perms, starts))
