"""Pins of the oracle's joint search over order and batch sizes (squeeze / delay moves of
Algorithm 1, batch-size sequence of the Problem Formulation) against values and facts that
do not come from it.

- hand-worked timelines with unequal batch sizes, every (order, layout) of a 3-request
  queue, and the joint optimum (tests/golden/worked_batch_sizes.json);
- special cases that reduce to the independently pinned fixed-size replay: maximum-size
  layouts are the static policy at that batch size, all-ones layouts are batch size 1;
- within-batch order invariance, move validity and move inverses;
- the exhaustive search against an enumeration written here with itertools.
"""
import itertools
import json
import os

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from paper_2504_14966_amd.workloads import Model, Queue, random_queue

GOLD = os.path.join(os.path.dirname(__file__), "golden", "worked_batch_sizes.json")
SEARCH = 2  # static admission with searched batch sizes


def _gold():
    with open(GOLD) as f:
        return json.load(f)


def _gold_queue(g):
    q = g["queue"]
    return Queue(np.array(q["in_len"], np.uint16), np.array(q["out_len"], np.uint16),
                 np.array(q["kind"], np.uint8), np.array(q["thr_us"], np.uint32))


def _gold_model(g, B=None):
    return Model(B or g["max_batch"], SEARCH, **g["model"])


def _key(s):
    a, b = s.split("|")
    return [int(x) for x in a.split(",")], [int(x) for x in b.split(",")]


def test_worked_detail(orc):
    g = _gold()
    q, m = _gold_queue(g), _gold_model(g)
    for case in g["detail"]:
        n, t, ttft, e2e = orc.replay_batches(q, m, case["perm"], case["starts"], detail=True)
        assert (n, t) == (case["n"], case["t"]), case["perm"]
        assert ttft.tolist() == case["ttft"] and e2e.tolist() == case["e2e"], case["perm"]


def test_worked_all_pairs_and_joint_optimum(orc):
    g = _gold()
    q, m = _gold_queue(g), _gold_model(g)
    for k, v in g["all"].items():
        perm, starts = _key(k)
        assert list(orc.replay_batches(q, m, perm, starts)) == v, k
    bn, bt, bp, bs, cnt = orc.brute_batches(q, m)
    opt = g["optimum"]
    assert [bn, bt] == opt["key"]
    assert bp.tolist() == opt["first_perm"] and bs.tolist() == opt["first_starts"]
    assert cnt == opt["count"]
    # the fixed-size optimum (every batch at the maximum) is strictly worse here
    fixed = Model(g["max_batch"], 0, **g["model"])
    fn, ft, _, _ = orc.brute(q, fixed)
    assert [fn, ft] == opt["max_size_layouts_only"]
    assert orc.better((bn, bt), (fn, ft))


def test_invalid_layouts(orc):
    g = _gold()
    q, m = _gold_queue(g), _gold_model(g)
    for starts in ([0, 1, 0], [1, 0, 0], [1, 2, 0]):   # no start at 0, run of 3 > 2, bad flag
        assert orc.replay_batches(q, m, [0, 1, 2], starts) == (-1, -1)
    assert orc.replay_batches(q, m, [0, 0, 2], [1, 1, 1]) == (-1, -1)
    assert not orc.check_starts([1, 0, 0], 3, 2) and orc.check_starts([1, 0, 0], 3, 3)


def test_worked_moves(orc):
    g = _gold()
    for c in g["moves"]["cases"]:
        f = orc.squeeze if c["move"] == "squeeze" else orc.delay
        made, p, s = f(c["perm"], c["starts"], c["B"], c["i"])
        assert made == c["made"], c
        if made:
            assert p.tolist() == c["perm_out"] and s.tolist() == c["starts_out"], c
        else:
            assert p.tolist() == c["perm"] and s.tolist() == c["starts"], c


def test_op3_thirds(orc):
    assert [orc.op3(w) for w in (0, 0x55555555, 0x55555556, 0xAAAAAAAA, 0xAAAAAAAB, 0xFFFFFFFF)] == [0, 0, 1, 1, 2, 2]


def _layout(rng, n, B):
    st = np.zeros(n, np.uint8)
    p = 0
    while p < n:
        st[p] = 1
        p += int(rng.integers(1, B + 1))
    return st


@settings(max_examples=60, deadline=None)
@given(n=st.integers(1, 40), B=st.integers(1, 9), seed=st.integers(0, 2**31))
def test_max_size_layout_is_static_policy(orc, n, B, seed):
    rng = np.random.default_rng(seed)
    q = random_queue(np.random.default_rng(seed + 1), n)
    m = Model(B, SEARCH, 2000, 40, 8000, 300, 2)
    ms = Model(B, 0, 2000, 40, 8000, 300, 2)
    perm = rng.permutation(n).astype(np.uint16)
    st_max = orc.max_starts(n, B)
    assert st_max.tolist() == [int(p % B == 0) for p in range(n)]
    got = orc.replay_batches(q, m, perm, st_max, detail=True)
    want = orc.replay(q, ms, perm, detail=True)
    assert got[:2] == want[:2]
    assert np.array_equal(got[2], want[2]) and np.array_equal(got[3], want[3])
    # the fixed-size replay treats the search policy as static
    assert orc.replay(q, m, perm) == want[:2]
    # batch size 1 everywhere is the static policy at B = 1, whatever the maximum
    ones = np.ones(n, np.uint8)
    assert orc.replay_batches(q, m, perm, ones) == orc.replay(q, Model(1, 0, 2000, 40, 8000, 300, 2), perm)


@settings(max_examples=60, deadline=None)
@given(n=st.integers(2, 40), B=st.integers(1, 9), seed=st.integers(0, 2**31))
def test_within_batch_order_free(orc, n, B, seed):
    rng = np.random.default_rng(seed)
    q = random_queue(np.random.default_rng(seed + 1), n)
    m = Model(B, SEARCH, 2000, 40, 8000, 300, 2)
    perm = rng.permutation(n).astype(np.uint16)
    starts = _layout(rng, n, B)
    base = orc.replay_batches(q, m, perm, starts)
    bounds = list(np.flatnonzero(starts)) + [n]
    p2 = perm.copy()
    for a, b in zip(bounds[:-1], bounds[1:]):
        p2[a:b] = rng.permutation(p2[a:b])
    assert orc.replay_batches(q, m, p2, starts) == base


@settings(max_examples=80, deadline=None)
@given(n=st.integers(1, 30), B=st.integers(1, 8), seed=st.integers(0, 2**31))
def test_moves_keep_valid_layouts(orc, n, B, seed):
    rng = np.random.default_rng(seed)
    perm = rng.permutation(n).astype(np.uint16)
    starts = _layout(rng, n, B)
    for _ in range(40):
        i = int(rng.integers(0, n))
        f = orc.squeeze if rng.integers(0, 2) else orc.delay
        made, p2, s2 = f(perm, starts, B, i)
        assert orc.check_starts(s2, n, B)
        assert sorted(p2.tolist()) == list(range(n))
        if made:
            # an allowed move always changes the layout
            assert not np.array_equal(s2, starts)
            perm, starts = p2, s2
        else:
            assert np.array_equal(s2, starts) and np.array_equal(p2, perm)


@settings(max_examples=60, deadline=None)
@given(n=st.integers(3, 30), B=st.integers(2, 8), seed=st.integers(0, 2**31))
def test_delay_undoes_squeeze(orc, n, B, seed):
    """A request squeezed out of a batch of two or more, then delayed, is back in its batch:
    same layout, same batch contents, same score."""
    rng = np.random.default_rng(seed)
    q = random_queue(np.random.default_rng(seed + 1), n)
    m = Model(B, SEARCH, 2000, 40, 8000, 300, 2)
    perm = rng.permutation(n).astype(np.uint16)
    starts = _layout(rng, n, B)
    for i in range(n):
        s = max(p for p in range(i + 1) if starts[p])
        e = next((p for p in range(i + 1, n) if starts[p]), n)
        made, p2, s2 = orc.squeeze(perm, starts, B, i)
        if not made or e - s < 2:
            continue
        assert p2[s] == perm[i]
        made2, p3, s3 = orc.delay(p2, s2, B, s)
        assert made2 and np.array_equal(s3, starts)
        assert sorted(p3[s:e].tolist()) == sorted(perm[s:e].tolist())
        assert orc.replay_batches(q, m, p3, s3) == orc.replay_batches(q, m, perm, starts)


def _enumerate(orc, q, m):
    n, B = q.n, m.max_batch
    best, first, count = None, None, 0
    for perm in itertools.permutations(range(n)):
        for mask in range(1 << (n - 1)):
            starts = [1] + [(mask >> (u - 1)) & 1 for u in range(1, n)]
            if not orc.check_starts(starts, n, B):
                continue
            k = orc.replay_batches(q, m, perm, starts)
            if best is None or orc.better(k, best):
                best, first, count = k, (list(perm), starts), 1
            elif k == best:
                count += 1
    return best, first, count


@pytest.mark.parametrize("n,B,seed", [(4, 2, 1), (5, 3, 2), (5, 2, 3), (6, 4, 4), (6, 6, 5)])
def test_brute_matches_enumeration(orc, n, B, seed):
    q = random_queue(np.random.default_rng(seed + 1), n)
    m = Model(B, SEARCH, 2000, 40, 8000, 300, 2)
    bn, bt, bp, bs, cnt = orc.brute_batches(q, m)
    best, first, count = _enumerate(orc, q, m)
    assert (bn, bt) == tuple(best)
    assert (bp.tolist(), bs.tolist()) == (first[0], first[1])
    assert cnt == count
    # never worse than the best max-size layout, and equal to brute force at batch size 1
    fn, ft, _, _ = orc.brute(q, Model(B, 0, 2000, 40, 8000, 300, 2))
    assert not orc.better((fn, ft), (bn, bt))
    if B == 1:
        assert (bn, bt) == (fn, ft)


def test_brute_batch_size_one(orc):
    q = random_queue(np.random.default_rng(11), 6)
    m = Model(1, SEARCH, 2000, 40, 8000, 300, 2)
    bn, bt, bp, bs, cnt = orc.brute_batches(q, m)
    fn, ft, fp, fc = orc.brute(q, Model(1, 0, 2000, 40, 8000, 300, 2))
    assert (bn, bt, bp.tolist(), cnt) == (fn, ft, fp.tolist(), fc)
    assert bs.tolist() == [1] * 6


# ---- the annealing chain of the joint search (trajectory: parity unpinned; properties) ----

def _energy(k, t_ref):
    return k[0] * t_ref - k[1]


@pytest.mark.parametrize("seed", range(4))
def test_chain_zero_temperature_is_greedy(orc, seed):
    rng = np.random.default_rng(seed)
    q = random_queue(rng, 12, max_in=1500, max_out=30, thr_hi=600_000)
    m = Model(3, SEARCH, p0=2000, p1=40, d0=8000, d1=300, d2=2)
    info = orc.start(q, m)
    res = orc.anneal_chain_batches(q, m, chain=seed, iters=400, T0=1e-300, alpha=0.5, seed=123, start_info=info,
                                   trace=True)
    e_prev = _energy((info[3], info[4]), info[1])
    for acc, n, t, _ in res["trace"]:
        e = _energy((n, t), info[1])
        assert e >= e_prev
        e_prev = e


@pytest.mark.parametrize("n,B,seed", [(12, 3, 0), (20, 4, 1), (9, 9, 2), (7, 1, 3)])
def test_chain_records_are_consistent(orc, n, B, seed):
    rng = np.random.default_rng(seed)
    q = random_queue(rng, n, max_in=1500, max_out=30, thr_hi=900_000)
    m = Model(B, SEARCH, p0=2000, p1=40, d0=8000, d1=300, d2=2)
    info = orc.start(q, m)
    res = orc.anneal_chain_batches(q, m, seed, 1500, 1.0, 0.999, 7, start_info=info, trace=True)
    rec, tr = res["rec"], res["trace"]
    for p, s in (("cur", "cur_starts"), ("best", "best_starts")):
        assert sorted(res[p].tolist()) == list(range(n)) and orc.check_starts(res[s], n, B)
    assert orc.replay_batches(q, m, res["cur"], res["cur_starts"]) == (rec[0], rec[1])
    assert orc.replay_batches(q, m, res["best"], res["best_starts"]) == (rec[2], rec[3])
    assert rec[5] == tr[:, 0].sum()
    # moves that are not allowed are never accepted and change nothing
    blocked = tr[:, 3] >= 4
    assert not tr[blocked, 0].any()
    for k in np.flatnonzero(blocked):
        prev = (info[3], info[4]) if k == 0 else (tr[k - 1, 1], tr[k - 1, 2])
        assert (tr[k, 1], tr[k, 2]) == prev
    # the three moves are drawn uniformly
    ops = tr[:, 3] & 3
    for op in range(3):
        assert 0.27 < (ops == op).mean() < 0.40
    if B == 1:
        # batch size 1: squeeze and delay are never allowed
        assert set(tr[ops < 2, 3].tolist()) <= {4, 5}
    keys = [(info[3], info[4])] + [(int(a), int(b)) for acc, a, b, _ in tr if acc]
    assert (rec[2], rec[3]) == max(keys, key=lambda k: (k[0], -k[1]))


def test_chain_reaches_joint_optimum(orc):
    """The worked queue: the joint optimum (3, 132036) needs a batch of one; max-size
    batches reach only 2 SLOs."""
    g = _gold()
    q, m = _gold_queue(g), _gold_model(g)
    res = orc.anneal_chain_batches(q, m, 0, 300, 1.0, 0.99, 0)
    assert [res["rec"][2], res["rec"][3]] == g["optimum"]["key"]
    rng = np.random.default_rng(5)
    q = random_queue(rng, 6, max_in=1500, max_out=30, thr_hi=300_000)
    m = Model(3, SEARCH, p0=2000, p1=40, d0=8000, d1=300, d2=2)
    bn, bt, *_ = orc.brute_batches(q, m)
    best = max(((r["rec"][2], r["rec"][3]) for r in
                (orc.anneal_chain_batches(q, m, c, 3000, 1.0, 0.998, 1) for c in range(4))),
               key=lambda k: (k[0], -k[1]))
    assert best == (bn, bt)


def test_chain_is_deterministic_and_chain_keyed(orc):
    rng = np.random.default_rng(9)
    q = random_queue(rng, 16, max_in=1500, max_out=30)
    m = Model(4, SEARCH, p0=2000, p1=40, d0=8000, d1=300, d2=2)
    info = orc.start(q, m)
    a = orc.anneal_chain_batches(q, m, 3, 300, 1.0, 0.999, 5, start_info=info)
    b = orc.anneal_chain_batches(q, m, 3, 300, 1.0, 0.999, 5, start_info=info)
    c = orc.anneal_chain_batches(q, m, 4, 300, 1.0, 0.999, 5, start_info=info)
    assert a["rec"].tolist() == b["rec"].tolist() and a["cur_starts"].tolist() == b["cur_starts"].tolist()
    assert a["rec"][6] != c["rec"][6]


def test_chain_single_request(orc):
    q = Queue(np.array([10], np.uint16), np.array([3], np.uint16), np.array([2], np.uint8),
              np.array([10**6], np.uint32))
    m = Model(4, SEARCH, p0=2000, p1=40, d0=8000, d1=300, d2=2)
    res = orc.anneal_chain_batches(q, m, 0, 50, 1.0, 0.99, 0, trace=True)
    assert res["rec"][5] == 0 and res["cur"].tolist() == [0] and res["cur_starts"].tolist() == [1]
