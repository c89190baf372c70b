"""Pins of the oracle's timeline replay against values and facts that do not come from it.

- hand-worked timelines (tests/golden/worked_timelines.json);
- closed forms: at batch size 1 a request's latency is its solo execution time plus the
  solo times of everything ahead of it (e2e = exec + wait, wait = sum of earlier batch
  durations, Section "Problem Formulation"); the solo time is the prefill plus the
  per-token decode time summed over the output tokens (Section "Latency Predictor"),
  whose arithmetic series has a closed form;
- static batches: an independent pairwise closed form of every member's finish offset;
- Smith's rule (1956): at batch size 1, ordering by shortest processing time minimises
  the sum of completion times, so brute force must find exactly that minimum;
- invariants of the batching model.
"""
import itertools
import json
import os

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from paper_2504_14966_amd.workloads import Model, Queue, random_queue

GOLD = os.path.join(os.path.dirname(__file__), "golden", "worked_timelines.json")


def _gold():
    with open(GOLD) as f:
        return json.load(f)


def _gold_queue(g):
    q = g["queue"]
    return Queue(np.array(q["in_len"], np.uint16), np.array(q["out_len"], np.uint16),
                 np.array(q["kind"], np.uint8), np.array(q["thr_us"], np.uint32))


def _model(g, B, policy):
    return Model(B, policy, **g["model"])


def test_worked_timelines(orc):
    g = _gold()
    q = _gold_queue(g)
    for case in g["cases"]:
        n, t, ttft, e2e = orc.replay(q, _model(g, case["max_batch"], case["policy"]), case["perm"], detail=True)
        assert (n, t) == (case["n"], case["t"]), case["name"]
        assert ttft.tolist() == case["ttft"], case["name"]
        assert e2e.tolist() == case["e2e"], case["name"]


@pytest.mark.parametrize("table,B,policy", [("static_b2", 2, 0), ("continuous_b2", 2, 1), ("b1", 1, 0), ("b1", 1, 1)])
def test_worked_all_orders_and_brute(orc, table, B, policy):
    g = _gold()
    q = _gold_queue(g)
    m = _model(g, B, policy)
    want = g["all_orders"][table]
    for key, val in want.items():
        perm = [int(x) for x in key.split(",")]
        assert list(orc.replay(q, m, perm)) == val, (table, perm)
    bn, bt, bp, cnt = orc.brute(q, m)
    assert [bn, bt] == g["all_orders"]["optimum"][table]
    # lexicographically first optimal order
    first = min(tuple(int(x) for x in k.split(",")) for k, v in want.items() if v == [bn, bt])
    assert tuple(bp.tolist()) == first
    assert cnt == sum(1 for v in want.values() if v == [bn, bt])


def test_worked_solo(orc):
    g = _gold()
    q = _gold_queue(g)
    m = _model(g, 1, 0)
    assert [orc.solo(q, m, r) for r in range(3)] == g["all_orders"]["solo"]


def solo_closed_form(q, m, r):
    """prefill + sum_{k=1..L} (d0 + d1*1 + d2*(l+k)) = prefill + L*(d0+d1+d2*l) + d2*L(L+1)/2."""
    l, L = int(q.in_len[r]), int(q.out_len[r])
    return m.p0 + m.p1 * l + L * (m.d0 + m.d1 + m.d2 * l) + m.d2 * L * (L + 1) // 2


def static_closed_form(q, m, perm):
    """Independent closed form of the static-batch timeline.

    Within a batch all members start decoding together after one prefill of
    P = sum(p0 + p1*l_j). Member m with L_m output tokens finishes after
    F_m = P + L_m*d0 + sum_j [d1*mu_j + d2*(l_j*mu_j + mu_j*(mu_j+1)/2)],
    mu_j = min(L_j, L_m): member j is in the batch for mu_j of m's decode steps, at the
    s-th of which it contributes l_j + s context tokens. The batch lasts max F; the
    next batch starts when it ends.
    """
    B, N = m.max_batch, q.n
    ttft = np.zeros(N, np.int64)
    e2e = np.zeros(N, np.int64)
    start = 0
    for b0 in range(0, N, B):
        mem = [int(r) for r in perm[b0:b0 + B]]
        P = sum(m.p0 + m.p1 * int(q.in_len[r]) for r in mem)
        F = {}
        for r in mem:
            Lm = int(q.out_len[r])
            acc = P + Lm * m.d0
            for j in mem:
                mu = min(int(q.out_len[j]), Lm)
                acc += m.d1 * mu + m.d2 * (int(q.in_len[j]) * mu + mu * (mu + 1) // 2)
            F[r] = acc
        for r in mem:
            ttft[r] = start + P
            e2e[r] = start + F[r]
        start += max(F.values())
    return ttft, e2e


def met_count(q, ttft, e2e):
    n = 0
    for r in range(q.n):
        k, thr = int(q.kind[r]), int(q.thr_us[r])
        if k == 0:
            n += ttft[r] <= thr
        elif k == 2:
            n += e2e[r] <= thr
        else:
            n += (e2e[r] - ttft[r]) <= thr * int(q.out_len[r])
    return int(n)


@settings(max_examples=60, deadline=None)
@given(st.integers(1, 12), st.integers(1, 16), st.integers(0, 2**31 - 1))
def test_static_matches_pairwise_closed_form(orc, n, B, seed):
    rng = np.random.default_rng(seed)
    q = random_queue(rng, n, max_in=2048, max_out=40)
    m = Model(B, 0, p0=int(rng.integers(0, 5000)), p1=int(rng.integers(0, 60)), d0=int(rng.integers(0, 9000)),
              d1=int(rng.integers(0, 400)), d2=int(rng.integers(0, 4)))
    perm = rng.permutation(n).astype(np.uint16)
    nn, tt, ttft, e2e = orc.replay(q, m, perm, detail=True)
    cttft, ce2e = static_closed_form(q, m, perm)
    assert ttft.tolist() == cttft.tolist()
    assert e2e.tolist() == ce2e.tolist()
    assert tt == int(ce2e.sum())
    assert nn == met_count(q, cttft, ce2e)


@settings(max_examples=40, deadline=None)
@given(st.integers(1, 10), st.integers(0, 2**31 - 1), st.sampled_from([0, 1]))
def test_batch_one_is_exec_plus_wait(orc, n, seed, policy):
    """B = 1: e2e_i = exec_i + sum of exec of everything ahead (both policies)."""
    rng = np.random.default_rng(seed)
    q = random_queue(rng, n, max_in=1500, max_out=30)
    m = Model(1, policy, p0=2000, p1=40, d0=8000, d1=300, d2=2)
    perm = rng.permutation(n).astype(np.uint16)
    _, t, ttft, e2e = orc.replay(q, m, perm, detail=True)
    clock = 0
    for r in perm:
        ex = solo_closed_form(q, m, int(r))
        assert orc.solo(q, m, int(r)) == ex
        assert ttft[r] == clock + m.p0 + m.p1 * int(q.in_len[r])
        clock += ex
        assert e2e[r] == clock
    assert t == int(e2e.sum())


@pytest.mark.parametrize("seed", range(6))
def test_smith_rule_batch_one(orc, seed):
    """Brute-force minimum total latency at B = 1 equals the shortest-processing-time order's."""
    rng = np.random.default_rng(100 + seed)
    n = 6
    q = random_queue(rng, n, max_in=1000, max_out=50)
    # thresholds of 0 make every request miss except impossible ones, so the brute-force
    # optimum is decided by total latency alone
    q.thr_us[:] = 0
    q.kind[:] = 2
    m = Model(1, 0, p0=2000, p1=40, d0=8000, d1=300, d2=2)
    ex = np.array([solo_closed_form(q, m, r) for r in range(n)], dtype=np.int64)
    spt = np.argsort(ex, kind="stable")
    want = int(sum((n - k) * ex[spt[k]] for k in range(n)))
    bn, bt, _, _ = orc.brute(q, m)
    assert bn == 0 and bt == want
    assert orc.replay(q, m, spt.astype(np.uint16))[1] == want


def _rand_case(seed, n, max_out=30):
    rng = np.random.default_rng(seed)
    q = random_queue(rng, n, max_in=1500, max_out=max_out)
    m = Model(int(rng.integers(1, n + 2)), int(rng.integers(0, 2)), p0=2000, p1=40, d0=8000, d1=300, d2=2)
    return rng, q, m


@settings(max_examples=40, deadline=None)
@given(st.integers(1, 10), st.integers(0, 2**31 - 1))
def test_invariants_range_and_identical_swap(orc, n, seed):
    rng, q, m = _rand_case(seed, n)
    perm = rng.permutation(n).astype(np.uint16)
    nn, tt = orc.replay(q, m, perm)
    assert 0 <= nn <= n
    assert tt > 0
    if n >= 2:
        # make two requests identical, then swapping them leaves the key unchanged
        a, b = rng.choice(n, 2, replace=False)
        for arr in (q.in_len, q.out_len, q.kind, q.thr_us):
            arr[b] = arr[a]
        k1 = orc.replay(q, m, perm)
        pa, pb = int(np.where(perm == a)[0][0]), int(np.where(perm == b)[0][0])
        k2 = orc.replay(q, m, orc.swap(perm, pa, pb))
        assert k1 == k2


@settings(max_examples=30, deadline=None)
@given(st.integers(1, 8), st.integers(0, 2**31 - 1))
def test_static_batch_at_least_n_is_order_free(orc, n, seed):
    rng, q, _ = _rand_case(seed, n)
    m = Model(n + int(rng.integers(0, 3)), 0, p0=2000, p1=40, d0=8000, d1=300, d2=2)
    keys = {orc.replay(q, m, rng.permutation(n).astype(np.uint16)) for _ in range(5)}
    assert len(keys) == 1


@settings(max_examples=30, deadline=None)
@given(st.integers(1, 10), st.integers(0, 2**31 - 1))
def test_continuous_equals_static_when_b1_or_b_ge_n_or_equal_outputs(orc, n, seed):
    rng, q, _ = _rand_case(seed, n)
    perm = rng.permutation(n).astype(np.uint16)
    for B in (1, n, n + 3):
        ks = orc.replay(q, Model(B, 0, p0=2000, p1=40, d0=8000, d1=300, d2=2), perm)
        kc = orc.replay(q, Model(B, 1, p0=2000, p1=40, d0=8000, d1=300, d2=2), perm)
        assert ks == kc
    # equal output lengths: every continuous batch drains at once, exactly like static
    q.out_len[:] = q.out_len[0]
    B = int(rng.integers(1, n + 1))
    ks = orc.replay(q, Model(B, 0, p0=2000, p1=40, d0=8000, d1=300, d2=2), perm, detail=True)
    kc = orc.replay(q, Model(B, 1, p0=2000, p1=40, d0=8000, d1=300, d2=2), perm, detail=True)
    assert ks[:2] == kc[:2]
    assert ks[2].tolist() == kc[2].tolist() and ks[3].tolist() == kc[3].tolist()


@settings(max_examples=30, deadline=None)
@given(st.integers(2, 12), st.integers(0, 2**31 - 1))
def test_static_within_batch_order_free(orc, n, seed):
    rng, q, _ = _rand_case(seed, n)
    B = int(rng.integers(1, n + 1))
    m = Model(B, 0, p0=2000, p1=40, d0=8000, d1=300, d2=2)
    perm = rng.permutation(n).astype(np.uint16)
    p2 = perm.copy()
    for b0 in range(0, n, B):
        p2[b0:b0 + B] = rng.permutation(p2[b0:b0 + B])
    assert orc.replay(q, m, perm) == orc.replay(q, m, p2)


def test_non_permutation_rows(orc):
    q = random_queue(np.random.default_rng(1), 5)
    m = Model(2, 0, p0=2000, p1=40, d0=8000, d1=300, d2=2)
    assert orc.replay(q, m, [0, 1, 2, 3, 3]) == (-1, -1)
    assert orc.replay(q, m, [0, 1, 2, 3, 5]) == (-1, -1)
    rows = np.array([[0, 1, 2, 3, 4], [4, 4, 4, 4, 4], [4, 3, 2, 1, 0]], np.uint16)
    out = orc.eval_rows(q, m, rows)
    assert out[1].tolist() == [-1, -1]
    assert out[0].tolist() == list(orc.replay(q, m, rows[0]))


def test_brute_matches_itertools_enumeration(orc):
    """The oracle's permutation enumeration finds the same optimum and count as itertools."""
    rng = np.random.default_rng(7)
    for n in (1, 2, 4, 6):
        q = random_queue(rng, n, max_in=500, max_out=20, thr_hi=400_000)
        for B, pol in ((1, 0), (2, 0), (3, 1)):
            m = Model(B, pol, p0=2000, p1=40, d0=8000, d1=300, d2=2)
            keys = {p: orc.replay(q, m, p) for p in itertools.permutations(range(n))}
            best = max(keys.values(), key=lambda k: (k[0], -k[1]))
            bn, bt, bp, cnt = orc.brute(q, m)
            assert (bn, bt) == best
            assert cnt == sum(1 for v in keys.values() if v == best)
            assert tuple(bp.tolist()) == min(p for p, v in keys.items() if v == best)
