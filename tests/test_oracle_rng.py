"""Pins of the oracle's random numbers, exponential and acceptance rule.

- Philox4x32-10 against the published known-answer vectors (tests/golden/philox_kat.json);
- det_exp against the C library exp: relative error bound, exact special points;
- the Metropolis rule: improvements always accepted; a worse candidate accepted with
  probability exp(delta / (t_ref * T)) (Section "Priority Mapping Algorithm": the
  higher the temperature, the likelier a worse solution is kept);
- proposal positions, the two moves and Fisher-Yates by their definitions.
"""
import json
import math
import os

import numpy as np
import pytest

KAT = os.path.join(os.path.dirname(__file__), "golden", "philox_kat.json")


def test_philox_known_answers(orc):
    with open(KAT) as f:
        vecs = json.load(f)["vectors"]
    for v in vecs:
        out = orc.philox([int(x, 16) for x in v["ctr"]], [int(x, 16) for x in v["key"]])
        assert [int(x) for x in out] == [int(x, 16) for x in v["out"]]


def _ulp_err(a, b):
    return abs(a - b) / math.ulp(b) if b != 0 else abs(a)


def test_det_exp_error_bound(orc):
    rng = np.random.default_rng(0)
    xs = np.concatenate([-rng.uniform(0, 708, 20000), -rng.uniform(0, 1, 5000), -rng.uniform(0, 1e-6, 1000),
                         -np.arange(0, 708, 0.25)])
    worst = 0.0
    for x in xs:
        worst = max(worst, _ulp_err(orc.det_exp(float(x)), math.exp(float(x))))
    assert worst <= 3.0, worst


def test_det_exp_special_points(orc):
    assert orc.det_exp(0.0) == 1.0
    assert orc.det_exp(-0.0) == 1.0
    assert orc.det_exp(-708.5) == 0.0
    assert orc.det_exp(-1e300) == 0.0
    assert orc.det_exp(float("-inf")) == 0.0
    assert orc.det_exp(-708.0) > 0.0
    # exp(-k ln2) = 2^-k; the rounded argument moves it by at most |x| * 2^-53 relative
    for k in range(1, 1000, 37):
        x = -k * math.log(2.0)
        y = orc.det_exp(x)
        assert _ulp_err(y, math.exp(x)) <= 3
        assert abs(y / 2.0 ** -k - 1.0) <= abs(x) * 2.0 ** -52 + 2.0 ** -50
    # monotone non-increasing as x decreases on a fine grid
    xs = np.linspace(-30, 0, 30001)
    ys = [orc.det_exp(float(x)) for x in xs]
    assert all(ys[i] <= ys[i + 1] for i in range(len(ys) - 1))


def test_accept_rule(orc):
    t_ref = 1_000_000
    for w3 in (0, 1, 2**31, 2**32 - 1):
        assert orc.accept(0, t_ref, 1.0, w3)          # equal score kept
        assert orc.accept(12345, t_ref, 1e-9, w3)     # improvement always kept
    # worse candidate: accepted iff u < exp(delta / (t_ref T)), away from the boundary
    rng = np.random.default_rng(3)
    for _ in range(3000):
        delta = -int(rng.integers(1, 5 * t_ref))
        T = float(rng.uniform(0.05, 3.0))
        w3 = int(rng.integers(0, 2**32))
        p = math.exp(delta / (t_ref * T))
        u = w3 / 2**32
        if abs(u - p) > 1e-9:
            assert orc.accept(delta, t_ref, T, w3) == (u < p)


def test_accept_frequency_matches_boltzmann(orc):
    """Sweeping u over [0,1) evenly, the accepted fraction is exp(delta/(t_ref T)); the paper's
    literal test (accept a worse move when exp(-(f_new-f)/T) < rand) would accept none."""
    t_ref = 10_000
    grid = np.arange(0, 2**32, 2**20, dtype=np.int64)
    for delta, T in ((-5000, 1.0), (-10000, 0.5), (-20000, 4.0)):
        frac = np.mean([orc.accept(delta, t_ref, T, int(w)) for w in grid])
        assert abs(frac - math.exp(delta / (t_ref * T))) < 2.0 / len(grid)


def test_positions_are_distinct_and_uniform(orc):
    n = 7
    counts = np.zeros((n, n), np.int64)
    rng = np.random.default_rng(5)
    for w1, w2 in rng.integers(0, 2**32, size=(21000, 2)):
        i, j = orc.positions(n, int(w1), int(w2))
        assert 0 <= i < n and 0 <= j < n and i != j
        counts[i, j] += 1
    off = counts[~np.eye(n, dtype=bool)]
    exp = 21000 / (n * (n - 1))
    chi2 = float(((off - exp) ** 2 / exp).sum())
    assert chi2 < 90  # 41 dof: p ~ 1e-5 cutoff
    assert orc.positions(1, 123, 456) == (0, 0)
    assert orc.positions(2, 0, 0) == (0, 1)
    assert orc.positions(2, 2**32 - 1, 2**32 - 1) == (1, 0)
    # extremes of multiply-shift
    assert orc.positions(1024, 2**32 - 1, 2**32 - 1) == (1023, 1022)


def test_moves_by_definition(orc):
    p = np.arange(6, dtype=np.uint16)
    assert orc.swap(p, 1, 4).tolist() == [0, 4, 2, 3, 1, 5]
    assert orc.insert(p, 1, 4).tolist() == [0, 2, 3, 4, 1, 5]
    assert orc.insert(p, 4, 1).tolist() == [0, 4, 1, 2, 3, 5]
    assert orc.insert(p, 0, 5).tolist() == [1, 2, 3, 4, 5, 0]
    assert orc.insert(p, 5, 0).tolist() == [5, 0, 1, 2, 3, 4]
    # insert puts the element at index j and keeps the others' relative order
    rng = np.random.default_rng(9)
    for _ in range(200):
        n = int(rng.integers(2, 40))
        q = rng.permutation(n).astype(np.uint16)
        i, j = (int(x) for x in rng.choice(n, 2, replace=False))
        r = orc.insert(q, i, j)
        assert r[j] == q[i]
        assert [x for x in r if x != q[i]] == [x for x in q if x != q[i]]


def test_fisher_yates(orc):
    for n in (1, 2, 5, 128, 1024):
        for idx in (0, 1, 77):
            p = orc.fy_perm(0, n, idx)
            assert sorted(p.tolist()) == list(range(n))
    assert orc.fy_perm(0, 128, 3).tolist() == orc.fy_perm(0, 128, 3).tolist()
    assert orc.fy_perm(0, 128, 3).tolist() != orc.fy_perm(0, 128, 4).tolist()
    # all 24 orders of 4 items equally likely
    from collections import Counter
    c = Counter(tuple(orc.fy_perm(11, 4, k).tolist()) for k in range(24000))
    assert len(c) == 24
    chi2 = sum((v - 1000) ** 2 / 1000 for v in c.values())
    assert chi2 < 60  # 23 dof
