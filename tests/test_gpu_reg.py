"""GPU parity of the small-queue annealing kernels (order and request fields in registers,
at most 64 requests) against the oracle, bit for bit, per chain. Fixed-size batches of 1, 2,
4, 8 or 16: start order, records, final and best orders, and the cross-chain winner, for
every batch size, ragged queues, swap-only / insert-only / mixed moves and both objectives.
The joint order / batch-size search (layout as a register bit mask): records, orders and
layouts for batch sizes from 1 to 64 and both objectives."""
import os
import sys

import numpy as np
import pytest

sys.path.insert(0, os.path.dirname(__file__))
from gpu_helpers import oracle_chains  # noqa: E402

from paper_2504_14966_amd.workloads import Model, random_queue  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sl():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2504_14966_amd.sloanneal as m
    m.load_library()
    return m


def _run_check(sl, orc, q, m, chains, iters, T0, alpha, seed, search=None):
    import torch
    dq = sl.DeviceQueue.from_queue(q)
    ws = sl.sched_anneal(dq, m, chains, iters, T0, alpha, seed, search=sl.Search(*search) if search else None)
    rec, cur, best = sl.sched_chains(ws, q.n, chains, perms=True)
    st, info = sl.sched_start_info(ws, q.n)
    bp, key = sl.sched_best(ws, q.n)
    torch.cuda.synchronize()
    rec, cur, best = rec.cpu().numpy(), sl.as_u16(cur), sl.as_u16(best)
    s_orc = orc.Search(*search) if search else None
    oi = orc.start(q, m, s_orc)
    assert sl.as_u16(st).tolist() == oi[0].tolist()
    assert info.cpu().numpy().tolist() == [oi[1], oi[3], oi[4], int(oi[2])]
    want = oracle_chains(q, m, range(chains), iters, T0, alpha, seed, oi, search)
    for c in range(chains):
        wrec, wcur, wbest = want[c]
        assert rec[c].tolist() == wrec.tolist(), c
        assert cur[c].tolist() == wcur.tolist() and best[c].tolist() == wbest.tolist(), c
    if not (search and search[0]):
        k = max(range(chains), key=lambda c: (rec[c, 2], -rec[c, 3], -c))
        assert key.cpu().numpy().tolist() == [rec[k, 2], rec[k, 3], k]
        assert sl.as_u16(bp).tolist() == best[k].tolist()


@pytest.mark.parametrize("n,B", [(2, 1), (13, 1), (3, 2), (31, 2), (5, 4), (64, 4), (9, 8), (57, 8), (16, 16),
                                 (17, 16), (50, 16), (64, 16)])
@pytest.mark.parametrize("thr", [0, 1 << 32, 1 << 31])
def test_reg_kernel_shapes_and_moves(sl, orc, n, B, thr):
    rng = np.random.default_rng(n * 131 + B * 7 + (thr >> 30))
    q = random_queue(rng, n, max_in=3000, max_out=150, thr_hi=60_000 * n)
    m = Model(B, 0, p0=2000, p1=40, d0=8000, d1=300, d2=2, swap_threshold=thr)
    _run_check(sl, orc, q, m, 6, 400, 0.8, 0.995, 11)


def _static_narrow(q, m):
    # the fixed-size widths: every finish offset and doubled pair cost in 32 bits, 24-bit factors
    lmax, Lmax, b = int(q.in_len.max()), int(q.out_len.max()), min(q.n, m.max_batch)
    pf = m.p0 + m.p1 * lmax
    fmax = b * pf + Lmax * m.d0 + b * (m.d1 * Lmax + m.d2 * (lmax * Lmax + Lmax * (Lmax + 1) // 2))
    inner = 2 * (m.d1 + m.d2 * lmax) + m.d2 + m.d2 * Lmax
    return fmax < 2**32 - 1 and inner < 2**24 and m.d2 < 2**24 and b * Lmax * inner < 2**32 and m.d0 < 2**24


def _timeline_end(q, m):
    # the end of the timeline of any order and layout
    li, lo = q.in_len.astype(object), q.out_len.astype(object)
    return sum(m.p0 + m.p1 * li) + (m.d0 + m.d1) * sum(lo) + m.d2 * sum(lo * li + lo * (lo + 1) // 2)


@pytest.mark.parametrize("B,search", [(1, None), (16, None), (4, (1, 6, 1)), (8, (0, 4, 0))])
def test_reg_kernel_wide_timeline(sl, orc, B, search):
    # per-batch offsets within 32 bits but the whole timeline above 2^32: the batch starts
    # and the latency sum in 64 bits
    rng = np.random.default_rng(900 + B)
    q = random_queue(rng, 64, max_in=3000, max_out=250, thr_hi=4_000_000_000)
    m = Model(B, 0, p0=5_000_000, p1=100, d0=16_000_000, d1=1000, d2=3)
    assert _static_narrow(q, m) and _timeline_end(q, m) > 2**32
    _run_check(sl, orc, q, m, 6, 300, 2.0, 0.99, 21, search)


@pytest.mark.parametrize("n,B", [(65, 1), (100, 2), (128, 4), (129, 8), (150, 16), (192, 16), (177, 1), (70, 16)])
@pytest.mark.parametrize("thr", [0, 1 << 32, 1 << 31])
def test_reg_parts_shapes_and_moves(sl, orc, n, B, thr):
    # 65 to 192 requests: two or three positions per lane; swaps and inserts across parts
    rng = np.random.default_rng(n * 17 + B * 3 + (thr >> 30))
    q = random_queue(rng, n, max_in=3000, max_out=150, thr_hi=60_000 * n)
    m = Model(B, 0, p0=2000, p1=40, d0=8000, d1=300, d2=2, swap_threshold=thr)
    _run_check(sl, orc, q, m, 6, 300, 0.8, 0.995, 17)


@pytest.mark.parametrize("n,B,search", [(120, 8, (1, 20, 0)), (190, 16, (1, 7, 1)), (99, 4, (0, 5, 1))])
def test_reg_parts_objectives(sl, orc, n, B, search):
    rng = np.random.default_rng(300 + n + B)
    q = random_queue(rng, n, max_in=3000, max_out=150, thr_hi=6_000_000)
    m = Model(B, 0, p0=2000, p1=40, d0=8000, d1=300, d2=2)
    _run_check(sl, orc, q, m, 6, 400, 3.0, 0.97, 5, search)


@pytest.mark.parametrize("n,B", [(128, 16), (160, 4)])
def test_reg_parts_wide_timeline(sl, orc, n, B):
    rng = np.random.default_rng(910 + n + B)
    q = random_queue(rng, n, max_in=3000, max_out=250, thr_hi=4_000_000_000)
    m = Model(B, 0, p0=5_000_000, p1=100, d0=16_000_000, d1=1000, d2=3)
    assert _static_narrow(q, m) and _timeline_end(q, m) > 2**32
    _run_check(sl, orc, q, m, 6, 250, 2.0, 0.99, 29)


@pytest.mark.parametrize("B,search", [(8, (1, 20, 0)), (16, (1, 7, 1)), (4, (0, 5, 0)), (2, (1, 3, 1))])
def test_reg_kernel_objectives(sl, orc, B, search):
    rng = np.random.default_rng(200 + B)
    q = random_queue(rng, 48, max_in=3000, max_out=150, thr_hi=3_000_000)
    m = Model(B, 0, p0=2000, p1=40, d0=8000, d1=300, d2=2)
    _run_check(sl, orc, q, m, 8, 500, 3.0, 0.97, 5, search)


def _search_check(sl, orc, q, m, chains, iters, T0, alpha, seed, search=None):
    import torch
    sys.path.insert(0, os.path.dirname(__file__))
    from gpu_helpers import oracle_chains_batches
    dq = sl.DeviceQueue.from_queue(q)
    ws = sl.sched_anneal(dq, m, chains, iters, T0, alpha, seed, search=sl.Search(*search) if search else None)
    rec, cur, best = sl.sched_chains(ws, q.n, chains, perms=True)
    cs, bs, win = sl.sched_starts(ws, q.n, chains)
    torch.cuda.synchronize()
    rec, cur, best, cs, bs = rec.cpu().numpy(), sl.as_u16(cur), sl.as_u16(best), cs.cpu().numpy(), bs.cpu().numpy()
    s_orc = orc.Search(*search) if search else None
    info = orc.start(q, m, s_orc)
    want = oracle_chains_batches(q, m, range(chains), iters, T0, alpha, seed, info, search)
    for c in range(chains):
        w = want[c]
        assert rec[c].tolist() == w["rec"].tolist(), c
        assert cur[c].tolist() == w["cur"].tolist() and best[c].tolist() == w["best"].tolist(), c
        assert cs[c].tolist() == w["cur_starts"].tolist() and bs[c].tolist() == w["best_starts"].tolist(), c


@pytest.mark.parametrize("n,B", [(5, 2), (17, 5), (33, 16), (63, 9), (64, 32), (50, 64), (64, 1)])
def test_reg_search_shapes(sl, orc, n, B):
    # the joint order / batch-size search on small queues (layout as a register bit mask)
    rng = np.random.default_rng(500 + n * 3 + B)
    q = random_queue(rng, n, max_in=3000, max_out=150, thr_hi=60_000 * n)
    m = Model(B, 2, p0=2000, p1=40, d0=8000, d1=300, d2=2)
    _search_check(sl, orc, q, m, 6, 500, 0.8, 0.995, 13)


@pytest.mark.parametrize("n,B,search", [(64, 16, None), (50, 5, (1, 6, 1)), (64, 64, (0, 4, 0)), (33, 1, None)])
def test_reg_search_wide_timeline(sl, orc, n, B, search):
    # per-batch offsets within 32 bits, the whole timeline above 2^32: saturating prefix
    # sums and the exact latency sum
    rng = np.random.default_rng(950 + n + B)
    q = random_queue(rng, n, max_in=3000, max_out=250, thr_hi=4_000_000_000)
    m = Model(B, 2, p0=5_000_000, p1=100, d0=16_000_000 // max(1, B // 16), d1=1000, d2=3)
    assert _static_narrow(q, m) and _timeline_end(q, m) > 2**32
    _search_check(sl, orc, q, m, 6, 400, 2.0, 0.99, 23, search)


@pytest.mark.parametrize("n,B,search", [(24, 6, (1, 10, 1)), (48, 16, (1, 25, 0)), (40, 3, (0, 4, 1))])
def test_reg_search_objectives(sl, orc, n, B, search):
    rng = np.random.default_rng(600 + n + B)
    q = random_queue(rng, n, max_in=3000, max_out=150, thr_hi=3_000_000)
    m = Model(B, 2, p0=2000, p1=40, d0=8000, d1=300, d2=2)
    _search_check(sl, orc, q, m, 6, 600, 3.0, 0.97, 21, search)


@pytest.mark.parametrize("n,B,policy,search", [(17, 3, 0, None), (33, 7, 2, None), (64, 64, 0, None),
                                               (64, 16, 2, (1, 10, 1)), (30, 5, 0, (1, 6, 0)), (1, 4, 2, None)])
def test_reg_fit(sl, orc, n, B, policy, search):
    # the fitted model (Table 2) with the chat SLO on small queues: order, fields and layout
    # in registers; every member's time below 2^32 (the 32-bit replay)
    _reg_fit_check(sl, orc, n, B, policy, search, 1)


@pytest.mark.parametrize("n,B,policy,search", [(20, 4, 0, None), (64, 16, 2, (1, 8, 0)), (37, 64, 2, None)])
def test_reg_fit_wide_members(sl, orc, n, B, policy, search):
    # coefficients 64 times Table 2's: member times above 2^32, the 64-bit replay
    _reg_fit_check(sl, orc, n, B, policy, search, 64)


def _reg_fit_check(sl, orc, n, B, policy, search, scale):
    import torch
    from paper_2504_14966_amd.workloads import TABLE2_10NS
    rng = np.random.default_rng(700 + n + B + policy)
    q = random_queue(rng, n, max_in=2000, max_out=300, thr_hi=2_000_000_000)
    q.kind[::3] = 3
    thr2 = rng.integers(1_500_000, 1_800_000, n).astype(np.uint32) * (1 if scale == 1 else 40)
    coef = {k: v * scale for k, v in TABLE2_10NS.items()}
    fd, fo = sl.FitModel(B, policy, **coef), orc.FitModel(B, policy, **coef)
    big = max(int(coef["ap"]) * min(n, B) * int(a) + int(coef["bp"]) * min(n, B) + int(coef["cp"]) * int(a)
              + int(coef["dp"]) + int(L) * (int(coef["bd"]) * min(n, B) + int(coef["dd"]))
              + (int(coef["ad"]) * min(n, B) + int(coef["cd"])) * (int(L) * int(a) + int(L) * (int(L) + 1) // 2)
              for a, L in zip(q.in_len, q.out_len))
    assert (big < 2**32 - 1) == (scale == 1)
    dq = sl.DeviceQueue.from_queue(q)
    chains, iters = 6, 500
    ws = sl.sched_anneal_fit(dq, fd, chains, iters, 1.5, 0.98, 4, tpot_thr=sl.thr_to_device(thr2),
                             search=sl.Search(*search) if search else None)
    rec, cur, best = sl.sched_chains(ws, n, chains, perms=True)
    cs, bs, _ = sl.sched_starts(ws, n, chains)
    _, key = sl.sched_best(ws, n)
    torch.cuda.synchronize()
    rec, cur, best, cs, bs = rec.cpu().numpy(), sl.as_u16(cur), sl.as_u16(best), cs.cpu().numpy(), bs.cpu().numpy()
    s_orc = orc.Search(*search) if search else None
    info = orc.start_fit(q, fo, s_orc, thr2)
    for c in range(chains):
        w = orc.anneal_chain_fit(q, fo, c, iters, 1.5, 0.98, 4, search=s_orc, thr2=thr2, start_info=info)
        assert rec[c].tolist() == w["rec"].tolist(), c
        assert cur[c].tolist() == w["cur"].tolist() and best[c].tolist() == w["best"].tolist(), c
        assert cs[c].tolist() == w["cur_starts"].tolist() and bs[c].tolist() == w["best_starts"].tolist(), c
    if not (search and search[0]):
        k = max(range(chains), key=lambda c: (rec[c, 2], -rec[c, 3], -c))
        assert key.cpu().numpy().tolist() == [rec[k, 2], rec[k, 3], k]


@pytest.mark.parametrize("seed", range(24))
def test_reg_random_sweep(sl, orc, seed):
    # seeded random shapes across the register kernels' whole range: 1 to 192 requests, every
    # power-of-two batch size up to 16, narrow or wide timelines, any move mix, both objectives
    rng = np.random.default_rng(4000 + seed)
    n = int(rng.integers(1, 193))
    B = int(rng.choice([1, 2, 4, 8, 16]))
    thr = int(rng.choice([0, 1 << 31, 1 << 32, int(rng.integers(0, 1 << 32))]))
    if rng.random() < 0.3:
        q = random_queue(rng, n, max_in=3000, max_out=250, thr_hi=4_000_000_000)
        m = Model(B, 0, p0=5_000_000, p1=100, d0=16_000_000, d1=1000, d2=3, swap_threshold=thr)
    else:
        q = random_queue(rng, n, max_in=3000, max_out=150, thr_hi=60_000 * n)
        m = Model(B, 0, p0=2000, p1=40, d0=8000, d1=300, d2=2, swap_threshold=thr)
    assert _static_narrow(q, m)
    search = None if rng.random() < 0.5 else (1, int(rng.integers(1, 30)), int(rng.integers(0, 2)))
    _run_check(sl, orc, q, m, 4, 200, float(rng.choice([0.5, 2.0, 50.0])), 0.98, seed, search)


@pytest.mark.parametrize("seed", range(12))
def test_reg_search_random_sweep(sl, orc, seed):
    # the register search kernel over random shapes: 1 to 64 requests, maximum batch 1 to 64,
    # narrow or wide timelines, both objectives
    rng = np.random.default_rng(5000 + seed)
    n = int(rng.integers(1, 65))
    B = int(rng.integers(1, 65))
    if rng.random() < 0.3:
        q = random_queue(rng, n, max_in=3000, max_out=250, thr_hi=4_000_000_000)
        m = Model(B, 2, p0=5_000_000, p1=100, d0=16_000_000 // max(1, min(n, B) // 16 + 1), d1=1000, d2=3)
    else:
        q = random_queue(rng, n, max_in=3000, max_out=150, thr_hi=60_000 * n)
        m = Model(B, 2, p0=2000, p1=40, d0=8000, d1=300, d2=2)
    assert _static_narrow(q, m)
    search = None if rng.random() < 0.5 else (1, int(rng.integers(1, 30)), int(rng.integers(0, 2)))
    _search_check(sl, orc, q, m, 4, 250, float(rng.choice([0.5, 2.0, 50.0])), 0.98, seed, search)


@pytest.mark.parametrize("seed", range(8))
def test_fit_random_sweep(sl, orc, seed):
    # the fitted model over random shapes: 1 to 200 requests (register or window kernels),
    # both policies, member times below or above 2^32
    rng = np.random.default_rng(6000 + seed)
    n = int(rng.integers(1, 201))
    B = int(rng.integers(1, 33))
    policy = int(rng.choice([0, 2]))
    scale = int(rng.choice([1, 1, 64]))
    _reg_fit_sweep_case(sl, orc, rng, n, B, policy, scale, seed)


def _reg_fit_sweep_case(sl, orc, rng, n, B, policy, scale, seed):
    import torch
    from paper_2504_14966_amd.workloads import TABLE2_10NS
    q = random_queue(rng, n, max_in=2000, max_out=300, thr_hi=2_000_000_000)
    q.kind[::5] = 3
    thr2 = (rng.integers(1_500_000, 1_800_000, n) * scale).astype(np.uint32)
    coef = {k: v * scale for k, v in TABLE2_10NS.items()}
    fd, fo = sl.FitModel(B, policy, **coef), orc.FitModel(B, policy, **coef)
    dq = sl.DeviceQueue.from_queue(q)
    chains, iters = 4, 120
    ws = sl.sched_anneal_fit(dq, fd, chains, iters, 1.0, 0.98, seed, tpot_thr=sl.thr_to_device(thr2))
    rec, cur, best = sl.sched_chains(ws, n, chains, perms=True)
    cs, bs, _ = sl.sched_starts(ws, n, chains)
    torch.cuda.synchronize()
    rec, cur, best, cs, bs = rec.cpu().numpy(), sl.as_u16(cur), sl.as_u16(best), cs.cpu().numpy(), bs.cpu().numpy()
    info = orc.start_fit(q, fo, None, thr2)
    for c in range(chains):
        w = orc.anneal_chain_fit(q, fo, c, iters, 1.0, 0.98, seed, thr2=thr2, start_info=info)
        assert rec[c].tolist() == w["rec"].tolist(), c
        assert cur[c].tolist() == w["cur"].tolist() and best[c].tolist() == w["best"].tolist(), c
        assert cs[c].tolist() == w["cur_starts"].tolist() and bs[c].tolist() == w["best_starts"].tolist(), c
