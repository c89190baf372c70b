"""GPU parity at the sizes and launch configurations bench.py times for the extensions:
every chain runs, and sampled chains (replayed one by one by the oracle) must agree bit for
bit -- records, final and best orders and layouts."""
import os
import sys

import numpy as np
import pytest

sys.path.insert(0, os.path.dirname(__file__))
from gpu_helpers import oracle_chains, oracle_chains_batches  # noqa: E402

from paper_2504_14966_amd.workloads import (TABLE2_10NS, chat_code_queue_10ns, multi_workload,  # noqa: E402
                                            search_workload, workload)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sl():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2504_14966_amd.sloanneal as m
    m.load_library()
    return m


def _fetch(sl, ws, n, chains, layouts):
    import torch
    rec, cur, best = sl.sched_chains(ws, n, chains, perms=True)
    out = dict(rec=rec, cur=cur, best=best)
    if layouts:
        out["cs"], out["bs"], _ = sl.sched_starts(ws, n, chains)
    torch.cuda.synchronize()
    return {k: (sl.as_u16(v) if k in ("cur", "best") else v.cpu().numpy()) for k, v in out.items()}


@pytest.mark.parametrize("wl,sample", [(4, (0, 2047, 4095)), (2, (0, 1023))])
def test_search_workloads_full(sl, orc, wl, sample):
    W = search_workload(wl)
    dq = sl.DeviceQueue.from_queue(W.queue)
    ws = sl.sched_anneal(dq, W.model, W.chains, W.iters, W.T0, W.alpha, W.seed)
    res = _fetch(sl, ws, W.queue.n, W.chains, True)
    info = orc.start(W.queue, W.model)
    want = oracle_chains_batches(W.queue, W.model, sample, W.iters, W.T0, W.alpha, W.seed, info)
    for c in sample:
        w = want[c]
        assert res["rec"][c].tolist() == w["rec"].tolist(), c
        assert res["best"][c].tolist() == w["best"].tolist() and res["bs"][c].tolist() == w["best_starts"].tolist(), c
        assert res["cur"][c].tolist() == w["cur"].tolist() and res["cs"][c].tolist() == w["cur_starts"].tolist(), c


def test_paper_schedule_full(sl, orc):
    W = workload(2)
    iters = 100 * sl.sched_levels(500.0, 20.0, 0.95)
    dq = sl.DeviceQueue.from_queue(W.queue)
    search = (1, 100, 1)
    ws = sl.sched_anneal(dq, W.model, W.chains, iters, 500.0, 0.95, 0, search=sl.Search(*search))
    res = _fetch(sl, ws, W.queue.n, W.chains, False)
    s = orc.Search(*search)
    info = orc.start(W.queue, W.model, s)
    sample = (0, 777, 1023)
    want = oracle_chains(W.queue, W.model, sample, iters, 500.0, 0.95, 0, info, search)
    for c in sample:
        rec, cur, best = want[c]
        assert res["rec"][c].tolist() == rec.tolist() and res["best"][c].tolist() == best.tolist(), c


def test_multi_workload_full(sl, orc):
    import torch
    W = multi_workload()
    I = W.extra["instances"]
    dq = sl.DeviceQueue.from_queue(W.queue)
    inst = sl.sched_assign(dq, torch.tensor(W.extra["capacity"], dtype=torch.int64, device="cuda"))
    mws = sl.sched_anneal_multi(dq, W.model, inst, I, W.chains, W.iters, W.T0, W.alpha, W.seed)
    inst_h = inst.cpu().numpy()
    assert np.array_equal(inst_h, orc.assign(W.queue, I, W.extra["capacity"]))
    for k in (0, I - 1):
        sq, ids = orc.sub_queue(W.queue, inst_h, k)
        res = _fetch(sl, mws.instance(k), sq.n, W.chains, False)
        info = orc.start(sq, W.model)
        sample = (0, W.chains - 1)
        want = oracle_chains(sq, W.model, [k * W.chains + c for c in sample], W.iters, W.T0, W.alpha, W.seed, info)
        for c in sample:
            rec, cur, best = want[k * W.chains + c]
            assert res["rec"][c].tolist() == rec.tolist() and res["best"][c].tolist() == best.tolist(), (k, c)


def test_fit_chat_code_full(sl, orc):
    q, thr2 = chat_code_queue_10ns(256, 0)
    fd = sl.FitModel(16, 2, **TABLE2_10NS)
    fo = orc.FitModel(16, 2, **TABLE2_10NS)
    dq = sl.DeviceQueue.from_queue(q)
    ws = sl.sched_anneal_fit(dq, fd, 2048, 2000, 1.0, 0.999, 0, tpot_thr=sl.thr_to_device(thr2))
    res = _fetch(sl, ws, q.n, 2048, True)
    info = orc.start_fit(q, fo, None, thr2)
    for c in (0, 2047):
        w = orc.anneal_chain_fit(q, fo, c, 2000, 1.0, 0.999, 0, thr2=thr2, start_info=info)
        assert res["rec"][c].tolist() == w["rec"].tolist(), c
        assert res["best"][c].tolist() == w["best"].tolist() and res["bs"][c].tolist() == w["best_starts"].tolist(), c
