"""Pins of the oracle's fitted latency predictor taken literally (per-request prefill and
decode with the batch-size interaction terms, the paper's Table 2 coefficients) and of
the paper's chat SLO (TTFT and TPOT), against values and facts that do not come from it:

- hand-worked terms and timelines with Table 2 in units of 10 ns
  (tests/golden/worked_fit_model.json);
- the decode sum against its closed form;
- batch size 1: e2e are running sums of the solo times, and Smith's rule fixes the
  minimum total latency;
- the chat SLO reduces to the TTFT kind with an unbounded TPOT threshold and to the TPOT
  kind with an unbounded TTFT threshold; within-batch order invariance.
"""
import itertools
import json
import os

import numpy as np
import pytest

from paper_2504_14966_amd.workloads import Queue, random_queue

GOLD = os.path.join(os.path.dirname(__file__), "golden", "worked_fit_model.json")


def _gold():
    with open(GOLD) as f:
        return json.load(f)


def _q(g, kind=None, thr=None):
    q = g["queue"]
    return Queue(np.array(q["in_len"], np.uint16), np.array(q["out_len"], np.uint16),
                 np.array(kind if kind is not None else q["kind"], np.uint8),
                 np.array(thr if thr is not None else q["thr"], np.uint32))


def test_table2_terms(orc):
    g = _gold()
    fm = orc.FitModel(g["max_batch"], 0, **g["model_10ns"])
    assert g["model_10ns"] == orc.TABLE2_10NS
    for k, v in g["terms"]["prefill"].items():
        b, l = map(int, k.split(","))
        assert orc.fit_prefill(fm, b, l) == v, k
    for k, v in g["terms"]["decode"].items():
        b, l, L = map(int, k.split(","))
        assert orc.fit_decode(fm, b, l, L) == v, k


def test_worked_timelines(orc):
    g = _gold()
    q = _q(g)
    fm = orc.FitModel(g["max_batch"], 0, **g["model_10ns"])
    for c in g["cases"]:
        n, t, ttft, e2e = orc.replay_fit(q, fm, c["perm"], c["starts"], detail=True)
        assert (n, t) == (c["n"], c["t"]), c["perm"]
        assert ttft.tolist() == c["ttft"] and e2e.tolist() == c["e2e"], c["perm"]


def test_worked_dual_slo(orc):
    g = _gold()
    d = g["dual"]
    kind = list(g["queue"]["kind"])
    kind[0] = orc.KIND_TTFT_TPOT
    thr = list(g["queue"]["thr"])
    thr[0] = d["thr"]
    q = _q(g, kind, thr)
    fm = orc.FitModel(g["max_batch"], 0, **g["model_10ns"])
    for t2, want in ((d["thr2_missed"], d["n_missed"]), (d["thr2_met"], d["n_met"])):
        thr2 = np.zeros(3, np.uint32)
        thr2[0] = t2
        assert orc.replay_fit(q, fm, [0, 1, 2], None, thr2)[0] == want
    # the chat kind needs its second threshold array
    assert orc.replay_fit(q, fm, [0, 1, 2]) == (-1, -1)


@pytest.mark.parametrize("seed", range(20))
def test_decode_closed_form(orc, seed):
    rng = np.random.default_rng(seed)
    c = {k: int(rng.integers(0, 30000)) for k in ("ap", "bp", "cp", "dp", "ad", "bd", "cd", "dd")}
    fm = orc.FitModel(64, 0, **c)
    for _ in range(20):
        b, l, L = int(rng.integers(1, 65)), int(rng.integers(0, 8193)), int(rng.integers(1, 1025))
        want = L * (c["bd"] * b + c["dd"]) + (c["ad"] * b + c["cd"]) * (L * l + L * (L + 1) // 2)
        assert orc.fit_decode(fm, b, l, L) == want
        assert orc.fit_prefill(fm, b, l) == c["ap"] * b * l + c["bp"] * b + c["cp"] * l + c["dp"]


@pytest.mark.parametrize("seed", range(4))
def test_batch_size_one_and_smith(orc, seed):
    rng = np.random.default_rng(seed)
    q = random_queue(rng, 6, max_in=3000, max_out=60)
    fm = orc.FitModel(1, 0, **orc.TABLE2_10NS)
    solo = [orc.fit_prefill(fm, 1, int(q.in_len[r])) + orc.fit_decode(fm, 1, int(q.in_len[r]), int(q.out_len[r]))
            for r in range(q.n)]
    best = None
    for p in itertools.permutations(range(q.n)):
        n, t, ttft, e2e = orc.replay_fit(q, fm, p, detail=True)
        run = np.cumsum([solo[r] for r in p])
        assert [e2e[r] for r in p] == run.tolist()
        best = t if best is None else min(best, t)
    spt = sorted(range(q.n), key=lambda r: solo[r])
    assert orc.replay_fit(q, fm, spt)[1] == best


@pytest.mark.parametrize("seed", range(6))
def test_dual_kind_special_cases(orc, seed):
    rng = np.random.default_rng(seed)
    n, B = 30, 4
    q = random_queue(rng, n, max_in=3000, max_out=60, thr_hi=60_000_000)
    fm = orc.FitModel(B, 0, **orc.TABLE2_10NS)
    perm = rng.permutation(n)
    big = np.full(n, 0xFFFFFFFE, np.uint32)
    # TTFT kind == chat kind with an unbounded TPOT threshold
    qt = Queue(q.in_len, q.out_len, np.zeros(n, np.uint8), q.thr_us)
    qd = Queue(q.in_len, q.out_len, np.full(n, 3, np.uint8), q.thr_us)
    assert orc.replay_fit(qt, fm, perm) == orc.replay_fit(qd, fm, perm, None, big)
    # TPOT kind == chat kind with an unbounded TTFT threshold
    qp = Queue(q.in_len, q.out_len, np.ones(n, np.uint8), q.thr_us)
    qd2 = Queue(q.in_len, q.out_len, np.full(n, 3, np.uint8), big)
    assert orc.replay_fit(qp, fm, perm) == orc.replay_fit(qd2, fm, perm, None, q.thr_us)


@pytest.mark.parametrize("seed", range(6))
def test_within_batch_order_free_and_layouts(orc, seed):
    rng = np.random.default_rng(seed)
    n, B = 25, 5
    q = random_queue(rng, n, max_in=3000, max_out=60, thr_hi=60_000_000)
    q.kind[::4] = 3
    thr2 = rng.integers(1_500_000, 1_800_000, n).astype(np.uint32)
    fm = orc.FitModel(B, 0, **orc.TABLE2_10NS)
    perm = rng.permutation(n).astype(np.uint16)
    base = orc.replay_fit(q, fm, perm, None, thr2)
    assert base == orc.replay_fit(q, fm, perm, orc.max_starts(n, B), thr2)
    p2 = perm.copy()
    for a in range(0, n, B):
        p2[a:a + B] = rng.permutation(p2[a:a + B])
    assert orc.replay_fit(q, fm, p2, None, thr2) == base


@pytest.mark.parametrize("policy", [0, 2])
def test_fit_chain_properties(orc, policy):
    rng = np.random.default_rng(12)
    n, B = 20, 4
    q = random_queue(rng, n, max_in=3000, max_out=60, thr_hi=80_000_000)
    q.kind[::3] = 3
    thr2 = rng.integers(1_500_000, 1_800_000, n).astype(np.uint32)
    fm = orc.FitModel(B, policy, **orc.TABLE2_10NS)
    res = orc.anneal_chain_fit(q, fm, 3, 800, 1.0, 0.995, 4, thr2=thr2)
    rec = res["rec"]
    assert orc.replay_fit(q, fm, res["cur"], res["cur_starts"], thr2) == (rec[0], rec[1])
    assert orc.replay_fit(q, fm, res["best"], res["best_starts"], thr2) == (rec[2], rec[3])
    info = orc.start_fit(q, fm, None, thr2)
    assert not orc.better((info[3], info[4]), (rec[2], rec[3]))
    if policy == 0:
        assert res["cur_starts"].tolist() == orc.max_starts(n, B).tolist()
    cold = orc.anneal_chain_fit(q, fm, 3, 400, 1e-300, 0.5, 4, thr2=thr2)
    assert not orc.better((info[3], info[4]), (cold["rec"][0], cold["rec"][1]))   # greedy: never below the start
