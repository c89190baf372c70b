"""GPU parity of sched_anneal / sched_best / sched_chains / sched_start_info against the
CPU oracle: start order and constants, and per chain the final order, best order, keys,
best iteration, accept count and trajectory digest, all bit-exact. The four annealing
workloads run at their full chain counts and iterations; sampled chains are replayed by
the oracle one by one."""
import os
import sys

import numpy as np
import pytest

sys.path.insert(0, os.path.dirname(__file__))
from gpu_helpers import oracle_chains  # noqa: E402

from paper_2504_14966_amd.workloads import Model, Queue, random_queue, workload  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sl():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2504_14966_amd.sloanneal as m
    m.load_library()
    return m


def _run(sl, q, m, chains, iters, T0, alpha, seed):
    import torch
    dq = sl.DeviceQueue.from_queue(q)
    ws = sl.sched_anneal(dq, m, chains, iters, T0, alpha, seed)
    rec, cur, best = sl.sched_chains(ws, q.n, chains, perms=True)
    st, info = sl.sched_start_info(ws, q.n)
    bp, key = sl.sched_best(ws, q.n)
    torch.cuda.synchronize()
    return dict(rec=rec.cpu().numpy(), cur=sl.as_u16(cur), best=sl.as_u16(best), start=sl.as_u16(st),
                info=info.cpu().numpy(), best_perm=sl.as_u16(bp), key=key.cpu().numpy(), ws=ws)


def _check(orc, res, q, m, sample, iters, T0, alpha, seed):
    info = orc.start(q, m)
    assert res["start"].tolist() == info[0].tolist()
    assert res["info"].tolist() == [info[1], info[3], info[4], int(info[2])]
    want = oracle_chains(q, m, sample, iters, T0, alpha, seed, info)
    for c in sample:
        rec, cur, best = want[c]
        assert res["rec"][c].tolist() == rec.tolist(), f"chain {c}"
        assert res["cur"][c].tolist() == cur.tolist(), f"chain {c}"
        assert res["best"][c].tolist() == best.tolist(), f"chain {c}"
    # the reduction: lexicographic argmax over all chains, lowest id on ties
    r = res["rec"]
    k = max(range(len(r)), key=lambda c: (r[c, 2], -r[c, 3], -c))
    assert res["key"].tolist() == [r[k, 2], r[k, 3], k]
    assert res["best_perm"].tolist() == res["best"][k].tolist()
    # every chain's orders are permutations and its keys are their replays (sampled)
    for c in list(sample)[:4]:
        assert orc.replay(q, m, res["cur"][c]) == (r[c, 0], r[c, 1])
        assert orc.replay(q, m, res["best"][c]) == (r[c, 2], r[c, 3])


def _sample(chains, extra=8, seed=0, first=8):
    rng = np.random.default_rng(seed)
    s = set(range(min(chains, first))) | {chains - 1}
    rest = np.setdiff1d(np.arange(chains), sorted(s))
    s |= set(rng.choice(rest, size=min(extra, rest.size), replace=False).tolist())
    return sorted(s)


def test_workload_1(sl, orc):
    W = workload(1)
    res = _run(sl, W.queue, W.model, W.chains, W.iters, W.T0, W.alpha, W.seed)
    _check(orc, res, W.queue, W.model, [0], W.iters, W.T0, W.alpha, W.seed)
    bn, bt, _, _ = orc.brute(W.queue, W.model)
    assert res["key"][:2].tolist() == [bn, bt]


def test_workload_2_every_chain(sl, orc):
    """All 1024 chains of the 64-request workload, replayed one by one by the oracle."""
    W = workload(2)
    res = _run(sl, W.queue, W.model, W.chains, W.iters, W.T0, W.alpha, W.seed)
    _check(orc, res, W.queue, W.model, list(range(W.chains)), W.iters, W.T0, W.alpha, W.seed)


def test_workload_3_full(sl, orc):
    """Chains 0..63, the last chain and 64 seeded-random ones of the continuous workload."""
    W = workload(3)
    res = _run(sl, W.queue, W.model, W.chains, W.iters, W.T0, W.alpha, W.seed)
    sample = _sample(W.chains, extra=64, seed=3, first=64)
    assert len(sample) == 129
    _check(orc, res, W.queue, W.model, sample, W.iters, W.T0, W.alpha, W.seed)


def test_workload_4_full(sl, orc):
    """Chains 0..63, the last chain and 64 seeded-random ones of the burst workload."""
    W = workload(4)
    res = _run(sl, W.queue, W.model, W.chains, W.iters, W.T0, W.alpha, W.seed)
    sample = _sample(W.chains, extra=64, seed=4, first=64)
    assert len(sample) == 129
    _check(orc, res, W.queue, W.model, sample, W.iters, W.T0, W.alpha, W.seed)


@pytest.mark.parametrize("n,B,policy,thr", [(1, 1, 0, 1 << 31), (2, 3, 1, 1 << 31), (9, 3, 0, 0), (9, 3, 1, 1 << 32),
                                            (17, 5, 0, 1 << 31), (40, 40, 0, 1 << 31), (70, 6, 1, 3 << 30),
                                            (130, 64, 0, 1 << 30), (200, 13, 1, 1 << 31), (300, 33, 0, 1 << 31),
                                            (1000, 50, 0, 3 << 30)])
def test_random_small_chains(sl, orc, n, B, policy, thr):
    rng = np.random.default_rng(n * 31 + B)
    q = random_queue(rng, n, max_in=3000, max_out=120, thr_hi=50_000 * n)
    m = Model(B, policy, p0=2000, p1=40, d0=8000, d1=300, d2=2, swap_threshold=thr)
    chains, iters = 24, 700
    res = _run(sl, q, m, chains, iters, 0.5, 0.995, 99)
    _check(orc, res, q, m, list(range(chains)), iters, 0.5, 0.995, 99)


def test_zero_iterations_and_t_ref_override(sl, orc):
    W = workload(2)
    m = Model(W.model.max_batch, W.model.policy, W.model.p0, W.model.p1, W.model.d0, W.model.d1, W.model.d2,
              t_ref_us=123456)
    res = _run(sl, W.queue, m, 16, 0, 1.0, 0.9, 0)
    info = orc.start(W.queue, m)
    assert res["info"][0] == 123456
    assert (res["rec"][:, 4] == -1).all() and (res["rec"][:, 5] == 0).all()
    assert (res["cur"] == info[0][None]).all()
    res = _run(sl, W.queue, m, 16, 300, 1.0, 0.99, 7)
    _check(orc, res, W.queue, m, list(range(16)), 300, 1.0, 0.99, 7)


def test_run_twice_is_bit_identical(sl):
    W = workload(2)
    a = _run(sl, W.queue, W.model, 256, 2000, W.T0, W.alpha, 3)
    b = _run(sl, W.queue, W.model, 256, 2000, W.T0, W.alpha, 3)
    for k in ("rec", "cur", "best", "key"):
        assert np.array_equal(a[k], b[k])


def test_short_workspace(sl):
    import torch
    W = workload(1)
    dq = sl.DeviceQueue.from_queue(W.queue)
    ws = torch.empty(sl.ws_bytes(8, 4) - 1, dtype=torch.uint8, device="cuda")
    with pytest.raises(sl.SchedError) as e:
        sl.sched_anneal(dq, W.model, 4, 10, 1.0, 0.99, 0, ws=ws)
    assert e.value.code == sl.SCHED_ENOSPC
