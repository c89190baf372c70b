"""Pins of the oracle's instance assignment (Scheduling Solution section): hand-worked
assignments (tests/golden/worked_assignment.json) and properties -- round-robin under equal
capacities, and within every iteration between resets no instance takes more than its
capacity except by the one request that starts it."""
import json
import os

import numpy as np
import pytest

from paper_2504_14966_amd.workloads import Model, Queue, random_queue

GOLD = os.path.join(os.path.dirname(__file__), "golden", "worked_assignment.json")


def _queue_of_needs(need):
    n = len(need)
    return Queue(np.array([x - 1 for x in need], np.uint16), np.ones(n, np.uint16), np.zeros(n, np.uint8),
                 np.zeros(n, np.uint32))


def test_worked_assignments(orc):
    with open(GOLD) as f:
        g = json.load(f)
    for c in g["cases"]:
        q = _queue_of_needs(c["need"])
        got = orc.assign(q, len(c["capacity"]), c["capacity"])
        assert got.tolist() == c["inst"], c["name"]


@pytest.mark.parametrize("seed", range(20))
def test_assignment_properties(orc, seed):
    rng = np.random.default_rng(seed)
    I = int(rng.integers(1, 9))
    q = random_queue(rng, int(rng.integers(1, 300)), max_in=3000, max_out=500)
    cap = rng.integers(500, 20000, size=I).astype(np.int64)
    inst = orc.assign(q, I, cap)
    assert inst.min() >= 0 and inst.max() < I
    need = q.in_len.astype(np.int64) + q.out_len
    # replay the iterations: a request that does not fit the roomiest instance starts a new
    # one; within an iteration every assignment goes to a roomiest instance that fits
    rem = cap.copy()
    for r in range(q.n):
        k = int(inst[r])
        if rem.max() < need[r]:
            rem = cap.copy()
            assert rem[k] == rem.max() and k == int(np.argmax(rem))
        else:
            assert rem[k] == rem.max() and k == int(np.argmax(rem)) and rem[k] >= need[r]
        rem[k] -= need[r]


def test_equal_capacities_round_robin(orc):
    """Equal capacities and equal requests: each instance is the roomiest in turn."""
    q = _queue_of_needs([37] * 97)
    for I in (1, 2, 3, 8, 64):
        inst = orc.assign(q, I, [10**9] * I)
        assert inst.tolist() == [r % I for r in range(q.n)]


def test_instance_chain_is_the_single_queue_chain(orc):
    """Each instance's chain c is the single-queue chain on its requests with Philox chain
    index k * chains_per_instance + c; its orders are permutations of the instance's requests."""
    rng = np.random.default_rng(8)
    q = random_queue(rng, 40, max_in=1500, max_out=30, thr_hi=500_000)
    m = Model(4, 0, p0=2000, p1=40, d0=8000, d1=300, d2=2)
    inst = orc.assign(q, 3, [5000, 4000, 3000])
    seen = []
    for k in range(3):
        res = orc.anneal_instance(q, m, inst, k, 8, 5, 300, 1.0, 0.99, 7)
        sq, ids = orc.sub_queue(q, inst, k)
        assert sorted(res["cur"].tolist()) == list(range(sq.n)) and res["ids"].tolist() == ids.tolist()
        assert orc.replay(sq, m, res["best"]) == (res["rec"][2], res["rec"][3])
        seen += ids[res["best"]].tolist()
    assert sorted(seen) == list(range(q.n))
