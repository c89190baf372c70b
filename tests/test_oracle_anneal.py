"""Properties of the oracle's annealing chain and start rule (the trajectory itself has no
published values: parity unpinned; these checks fix what the paper and the rule imply).

- start (Algorithm 1 initialisation): ascending solo latency, stable; the input order
  wins only when strictly better; with batch size 1 and every SLO met by the sorted
  order, that order is optimal (Section "Priority Mapping Algorithm");
- a chain at vanishing temperature is a greedy descent: the energy never drops;
- the recorded keys, orders and counters agree with independent replays;
- on small queues a long chain reaches the brute-force optimum (Table 1 compares SA
  against exhaustive search).
"""
import json
import math
import os

import numpy as np
import pytest

from paper_2504_14966_amd.workloads import Model, Queue, random_queue, workload

GOLD = os.path.join(os.path.dirname(__file__), "golden", "worked_timelines.json")


def _gq():
    with open(GOLD) as f:
        g = json.load(f)
    q = g["queue"]
    return g, Queue(np.array(q["in_len"], np.uint16), np.array(q["out_len"], np.uint16),
                    np.array(q["kind"], np.uint8), np.array(q["thr_us"], np.uint32))


def test_start_rule_worked(orc):
    g, q = _gq()
    # B=1: solo 23006, 29212, 18702 -> sorted (2,0,1) with key (1, 131330); the input order
    # (0,1,2) has (2, 146144), strictly better, so it becomes the start
    m = Model(1, 0, **g["model"])
    st, t_ref, allmet, sn, stt = orc.start(q, m)
    assert st.tolist() == [0, 1, 2] and (sn, stt) == (2, 146144) and not allmet
    assert t_ref == 146144
    # static B=2: sorted (2,0,1) -> (0, 121832); input (3, 118950) better
    st, t_ref, allmet, sn, stt = orc.start(q, Model(2, 0, **g["model"]))
    assert st.tolist() == [0, 1, 2] and (sn, stt) == (3, 118950)
    # loosen r1's SLO so the sorted order meets all at B=1
    q2 = Queue(q.in_len.copy(), q.out_len.copy(), q.kind.copy(), q.thr_us.copy())
    q2.thr_us[:] = [50_000, 80_000, 9000]
    st, t_ref, allmet, sn, stt = orc.start(q2, m)
    assert allmet and st.tolist() == [2, 0, 1] and (sn, stt) == (3, 131330)
    # t_ref override
    st, t_ref, *_ = orc.start(q, Model(1, 0, t_ref_us=777, **g["model"]))
    assert t_ref == 777


def test_start_sort_is_stable(orc):
    q = Queue(np.array([10, 20, 10, 20, 10], np.uint16), np.array([5, 1, 5, 1, 5], np.uint16),
              np.zeros(5, np.uint8), np.zeros(5, np.uint32))
    st, *_ = orc.start(q, Model(2, 0, p0=2000, p1=40, d0=8000, d1=300, d2=2))
    # requests 1, 3 are short and tie; 0, 2, 4 tie; identity is not strictly better
    assert st.tolist() == [1, 3, 0, 2, 4]


@pytest.mark.parametrize("seed", range(5))
def test_allmet_sorted_order_is_optimal_at_b1(orc, seed):
    rng = np.random.default_rng(40 + seed)
    q = random_queue(rng, 6, max_in=800, max_out=20)
    q.kind[:] = 2
    q.thr_us[:] = 10**9
    m = Model(1, 0, p0=2000, p1=40, d0=8000, d1=300, d2=2)
    st, t_ref, allmet, sn, stt = orc.start(q, m)
    assert allmet
    bn, bt, _, _ = orc.brute(q, m)
    assert (sn, stt) == (bn, bt)


def _energy(k, t_ref):
    return k[0] * t_ref - k[1]


@pytest.mark.parametrize("seed", range(4))
def test_zero_temperature_is_greedy(orc, seed):
    rng = np.random.default_rng(seed)
    q = random_queue(rng, 12, max_in=1500, max_out=30, thr_hi=600_000)
    m = Model(3, seed % 2, p0=2000, p1=40, d0=8000, d1=300, d2=2)
    info = orc.start(q, m)
    res = orc.anneal_chain(q, m, chain=seed, iters=400, T0=1e-300, alpha=0.5, seed=123, start_info=info, trace=True)
    tr = res["trace"]
    e_prev = _energy((info[3], info[4]), info[1])
    for acc, n, t, _ in tr:
        e = _energy((n, t), info[1])
        assert e >= e_prev
        e_prev = e


@pytest.mark.parametrize("wl", [1])
def test_chain_records_are_consistent(orc, wl):
    W = workload(wl)
    q, m = W.queue, W.model
    info = orc.start(q, m)
    res = orc.anneal_chain(q, m, 0, W.iters, W.T0, W.alpha, W.seed, start_info=info, trace=True)
    rec, tr = res["rec"], res["trace"]
    assert sorted(res["cur"].tolist()) == list(range(q.n))
    assert sorted(res["best"].tolist()) == list(range(q.n))
    assert orc.replay(q, m, res["cur"]) == (rec[0], rec[1])
    assert orc.replay(q, m, res["best"]) == (rec[2], rec[3])
    assert rec[5] == tr[:, 0].sum()
    assert (tr[-1, 1], tr[-1, 2]) == (rec[0], rec[1])
    # best is the lexicographic maximum over start and every accepted state, first reached
    keys = [(info[3], info[4])] + [(int(n), int(t)) for a, n, t, _ in tr if a]
    best = max(keys, key=lambda k: (k[0], -k[1]))
    assert (rec[2], rec[3]) == best
    if rec[4] >= 0:
        acc_iters = [k for k in range(len(tr)) if tr[k, 0]]
        first = next(k for k in acc_iters if (tr[k, 1], tr[k, 2]) == best)
        assert rec[4] == first
    # replaying from the trace: rejected proposals keep the key
    for k in range(1, len(tr)):
        if not tr[k, 0]:
            assert (tr[k, 1], tr[k, 2]) == (tr[k - 1, 1], tr[k - 1, 2])
    # the move mix is about 50/50 at the default threshold
    assert 0.4 < tr[:, 3].mean() < 0.6


def test_chain_reaches_brute_force_optimum(orc):
    """Workload 1 (8 requests): the best of a 2000-iteration chain against all 40320 orders."""
    W = workload(1)
    bn, bt, _, _ = orc.brute(W.queue, W.model)
    res = orc.anneal_chain(W.queue, W.model, 0, W.iters, W.T0, W.alpha, W.seed)
    assert (res["rec"][2], res["rec"][3]) == (bn, bt)


def test_chain_is_deterministic_and_chain_keyed(orc):
    W = workload(1)
    info = orc.start(W.queue, W.model)
    a = orc.anneal_chain(W.queue, W.model, 3, 300, 1.0, 0.999, 5, start_info=info)
    b = orc.anneal_chain(W.queue, W.model, 3, 300, 1.0, 0.999, 5, start_info=info)
    c = orc.anneal_chain(W.queue, W.model, 4, 300, 1.0, 0.999, 5, start_info=info)
    assert a["rec"].tolist() == b["rec"].tolist() and a["cur"].tolist() == b["cur"].tolist()
    assert a["rec"][6] != c["rec"][6]


def test_swap_only_and_insert_only(orc):
    W = workload(1)
    for thr, want in ((1 << 32, 0), (0, 1)):
        m = Model(W.model.max_batch, W.model.policy, W.model.p0, W.model.p1, W.model.d0, W.model.d1, W.model.d2,
                  swap_threshold=thr)
        res = orc.anneal_chain(W.queue, m, 0, 200, 1.0, 0.999, 0, trace=True)
        assert set(res["trace"][:, 3].tolist()) == {want}


def test_hot_chain_accepts_more_than_cold(orc):
    W = workload(1)
    hot = orc.anneal_chain(W.queue, W.model, 0, 1000, 100.0, 1.0, 0)["rec"][5]
    cold = orc.anneal_chain(W.queue, W.model, 0, 1000, 1e-4, 1.0, 0)["rec"][5]
    assert hot > cold


def test_degenerate_single_request(orc):
    q = Queue(np.array([10], np.uint16), np.array([3], np.uint16), np.array([2], np.uint8),
              np.array([10**6], np.uint32))
    m = Model(4, 0, p0=2000, p1=40, d0=8000, d1=300, d2=2)
    res = orc.anneal_chain(q, m, 0, 50, 1.0, 0.99, 0)
    assert res["rec"][5] == 50 and res["cur"].tolist() == [0] and res["rec"][4] == -1
