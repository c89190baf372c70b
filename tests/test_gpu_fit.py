"""GPU parity of the fitted latency model taken literally (per-request prefill and decode
with the batch-size interaction terms, Table 2 coefficients) and of the paper's chat SLO,
against the oracle, bit for bit: sched_eval_fit (with and without layouts, invalid rows)
and sched_anneal_fit per chain for fixed-size batches and the batch-size search."""
import os
import sys

import numpy as np
import pytest

sys.path.insert(0, os.path.dirname(__file__))

from paper_2504_14966_amd.workloads import TABLE2_10NS, Queue, chat_code_queue_10ns, random_layouts, random_queue  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sl():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2504_14966_amd.sloanneal as m
    m.load_library()
    return m


def _models(sl, orc, B, policy, coef=TABLE2_10NS):
    return sl.FitModel(B, policy, **coef), orc.FitModel(B, policy, **coef)


@pytest.mark.parametrize("n,B,seed", [(1, 4, 0), (3, 2, 1), (64, 16, 2), (128, 16, 3), (1000, 64, 4), (257, 33, 5)])
def test_eval_fit(sl, orc, n, B, seed):
    import torch
    rng = np.random.default_rng(seed)
    q = random_queue(rng, n, max_in=4000, max_out=600, thr_hi=3_000_000_000)
    q.kind[::3] = 3
    thr2 = rng.integers(1_500_000, 1_800_000, n).astype(np.uint32)
    fd, fo = _models(sl, orc, B, 2)
    k = 40
    perms = np.stack([rng.permutation(n) for _ in range(k)]).astype(np.uint16)
    starts = random_layouts(rng, k, n, B)
    starts[1] = orc.max_starts(n, B)
    if n > 2:
        perms[2, 0] = perms[2, 1]
        starts[3, 0] = 0
    dq = sl.DeviceQueue.from_queue(q)
    t2 = sl.thr_to_device(thr2)
    out, det = sl.sched_eval_fit(dq, fd, sl.perms_to_device(perms), sl.starts_to_device(starts), t2, detail=True)
    plain = sl.sched_eval_fit(dq, fd, sl.perms_to_device(perms), None, t2)
    torch.cuda.synchronize()
    out, det, plain = out.cpu().numpy(), det.cpu().numpy(), plain.cpu().numpy()
    for r in range(k):
        nn, tt, ttft, e2e = orc.replay_fit(q, fo, perms[r], starts[r], thr2, detail=True)
        assert out[r].tolist() == [nn, tt], r
        if nn >= 0:
            assert det[r, :, 0].tolist() == ttft.tolist() and det[r, :, 1].tolist() == e2e.tolist(), r
        assert plain[r].tolist() == list(orc.replay_fit(q, fo, perms[r], None, thr2)), r


def test_eval_fit_worked_and_rejections(sl, orc):
    import ctypes as C
    import json
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "worked_fit_model.json")))
    gq = g["queue"]
    q = Queue(np.array(gq["in_len"], np.uint16), np.array(gq["out_len"], np.uint16), np.array(gq["kind"], np.uint8),
              np.array(gq["thr"], np.uint32))
    fd = sl.FitModel(g["max_batch"], 2, **g["model_10ns"])
    perms = np.array([c["perm"] for c in g["cases"]], np.uint16)
    starts = np.array([c["starts"] for c in g["cases"]], np.uint8)
    dq = sl.DeviceQueue.from_queue(q)
    out, det = sl.sched_eval_fit(dq, fd, sl.perms_to_device(perms), sl.starts_to_device(starts), detail=True)
    out, det = out.cpu().numpy(), det.cpu().numpy()
    for r, c in enumerate(g["cases"]):
        assert out[r].tolist() == [c["n"], c["t"]]
        assert det[r, :, 0].tolist() == c["ttft"] and det[r, :, 1].tolist() == c["e2e"]
    # the chat kind needs the second threshold array
    # (checked on the device: every row reads (-2, SCHED_EINVAL))
    q3 = Queue(q.in_len, q.out_len, np.array([3, 2, 1], np.uint8), q.thr_us)
    bad = sl.sched_eval_fit(sl.DeviceQueue.from_queue(q3), fd, sl.perms_to_device(perms)).cpu().tolist()
    assert bad == [[-2, sl.SCHED_EINVAL]] * len(perms)
    L = sl.load_library()
    bad = sl.FitModel(2, 1, **g["model_10ns"])   # continuous admission is not a fitted-model policy
    qq = dq.c()
    assert L.sched_eval_fit(C.byref(qq), C.byref(bad), None, 8, None, 1, 8, None, None) == sl.SCHED_EINVAL


def _anneal(sl, q, fd, chains, iters, T0, alpha, seed, thr2, search):
    import torch
    dq = sl.DeviceQueue.from_queue(q)
    t2 = sl.thr_to_device(thr2) if thr2 is not None else None
    ws = sl.sched_anneal_fit(dq, fd, chains, iters, T0, alpha, seed, tpot_thr=t2,
                             search=sl.Search(*search) if search else None)
    rec, cur, best = sl.sched_chains(ws, q.n, chains, perms=True)
    cs, bs, win = sl.sched_starts(ws, q.n, chains)
    st, info = sl.sched_start_info(ws, q.n)
    bp, key = sl.sched_best(ws, q.n)
    torch.cuda.synchronize()
    return dict(rec=rec.cpu().numpy(), cur=sl.as_u16(cur), best=sl.as_u16(best), cs=cs.cpu().numpy(),
                bs=bs.cpu().numpy(), start=sl.as_u16(st), info=info.cpu().numpy(), key=key.cpu().numpy())


def _check_winner(res, ratio):
    # the cross-chain winner: best key by the objective, lowest chain on ties
    from fractions import Fraction
    r = res["rec"]
    if ratio:
        k = 0
        for c in range(1, len(r)):
            if Fraction(int(r[c, 2]), int(r[c, 3])) > Fraction(int(r[k, 2]), int(r[k, 3])):
                k = c
    else:
        k = max(range(len(r)), key=lambda c: (r[c, 2], -r[c, 3], -c))
    assert res["key"].tolist() == [r[k, 2], r[k, 3], k]


@pytest.mark.parametrize("policy,search", [(0, None), (2, None), (0, (1, 10, 0)), (2, (1, 10, 1))])
def test_anneal_fit_chat_code(sl, orc, policy, search):
    q, thr2 = chat_code_queue_10ns(64, 0)
    fd, fo = _models(sl, orc, 16, policy)
    chains, iters = 48, 600
    res = _anneal(sl, q, fd, chains, iters, 1.0, 0.995, 2, thr2, search)
    s_orc = orc.Search(*search) if search else None
    info = orc.start_fit(q, fo, s_orc, thr2)
    assert res["start"].tolist() == info[0].tolist()
    assert res["info"].tolist() == [info[1], info[3], info[4], int(info[2])]
    for c in range(0, chains, 5):
        w = orc.anneal_chain_fit(q, fo, c, iters, 1.0, 0.995, 2, search=s_orc, thr2=thr2, start_info=info)
        assert res["rec"][c].tolist() == w["rec"].tolist(), c
        assert res["cur"][c].tolist() == w["cur"].tolist() and res["best"][c].tolist() == w["best"].tolist(), c
        assert res["cs"][c].tolist() == w["cur_starts"].tolist() and res["bs"][c].tolist() == w["best_starts"].tolist(), c
    _check_winner(res, bool(search and search[0]))


@pytest.mark.parametrize("n,B,policy", [(1, 3, 0), (2, 1, 2), (40, 64, 2), (300, 8, 0)])
def test_anneal_fit_shapes(sl, orc, n, B, policy):
    rng = np.random.default_rng(n + B)
    q = random_queue(rng, n, max_in=4000, max_out=300, thr_hi=2_000_000_000)
    fd, fo = _models(sl, orc, B, policy)
    chains, iters = 8, 200
    res = _anneal(sl, q, fd, chains, iters, 0.5, 0.99, 7, None, None)
    info = orc.start_fit(q, fo)
    for c in range(chains):
        w = orc.anneal_chain_fit(q, fo, c, iters, 0.5, 0.99, 7, start_info=info)
        assert res["rec"][c].tolist() == w["rec"].tolist(), c
        assert res["best"][c].tolist() == w["best"].tolist(), c
    _check_winner(res, False)


@pytest.mark.parametrize("n,B,policy,scale", [(150, 16, 0, 1), (200, 16, 2, 1), (150, 16, 0, 64), (130, 33, 2, 64)])
def test_anneal_fit_windows_widths(sl, orc, n, B, policy, scale):
    # more than 64 requests (windows of whole batches): member times below 2^32 take the
    # 32-bit windows, above it the 64-bit ones
    from paper_2504_14966_amd.workloads import TABLE2_10NS
    rng = np.random.default_rng(n + B + scale)
    q = random_queue(rng, n, max_in=2000, max_out=300, thr_hi=2_000_000_000)
    q.kind[::4] = 3
    thr2 = (rng.integers(1_500_000, 1_800_000, n) * scale).astype(np.uint32)
    coef = {k: v * scale for k, v in TABLE2_10NS.items()}
    fd, fo = sl.FitModel(B, policy, **coef), orc.FitModel(B, policy, **coef)
    chains, iters = 6, 150
    res = _anneal(sl, q, fd, chains, iters, 1.0, 0.99, 3, thr2, None)
    info = orc.start_fit(q, fo, None, thr2)
    for c in range(chains):
        w = orc.anneal_chain_fit(q, fo, c, iters, 1.0, 0.99, 3, thr2=thr2, start_info=info)
        assert res["rec"][c].tolist() == w["rec"].tolist(), c
        assert res["cur"][c].tolist() == w["cur"].tolist() and res["best"][c].tolist() == w["best"].tolist(), c
        assert res["cs"][c].tolist() == w["cur_starts"].tolist() and res["bs"][c].tolist() == w["best_starts"].tolist(), c
    _check_winner(res, False)


@pytest.mark.parametrize("policy", [0, 2])
def test_fit_huge_times_batch_replay(sl, orc, policy):
    # member times of 2^56 and more: the windowed replay's keys would not hold them, so the
    # batch-at-a-time replay runs (its bound 2^57 <= timeline, timeline * (n + 2) < 2^62)
    import torch
    rng = np.random.default_rng(90 + policy)
    n, B = 3, 2
    q = random_queue(rng, n, max_in=1000, max_out=100, thr_hi=2**32 - 2)
    coef = dict(ap=3, bp=5, cp=7, dp=1 << 56, ad=1, bd=2, cd=3, dd=11)
    fd, fo = sl.FitModel(B, policy, **coef), orc.FitModel(B, policy, **coef)
    perms = np.stack([rng.permutation(n) for _ in range(12)]).astype(np.uint16)
    starts = random_layouts(rng, 12, n, B)
    dq = sl.DeviceQueue.from_queue(q)
    out = sl.sched_eval_fit(dq, fd, sl.perms_to_device(perms), sl.starts_to_device(starts))
    torch.cuda.synchronize()
    out = out.cpu().numpy()
    for r in range(12):
        assert out[r].tolist() == list(orc.replay_fit(q, fo, perms[r], starts[r])), r
    res = _anneal(sl, q, fd, 4, 50, 0.5, 0.99, 3, None, None)
    info = orc.start_fit(q, fo)
    for c in range(4):
        w = orc.anneal_chain_fit(q, fo, c, 50, 0.5, 0.99, 3, start_info=info)
        assert res["rec"][c].tolist() == w["rec"].tolist(), c
