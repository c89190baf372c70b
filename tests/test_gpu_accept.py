"""GPU parity of the acceptance step of Algorithm 1 as the annealing kernels evaluate it
(sched_accept_check): a single-precision screen decides most worse candidates and the
double-precision rule the rest. Every decision must equal the oracle's exact rule
(orc_accept / orc_accept_ratio: u < det_exp(x) in double), tolerance 0.

Inputs, about 1.2 million per rule, built in three groups:
- at the boundary: w3 within a few units of e^x * 2^32 (where only the double rule can
  decide, so the screen must step aside);
- at the screen's own edges: u placed so that log2(e^x / u) sits at +-0.9 .. 1.1 times the
  screen's threshold |xl| 2^-16 + 2^-10 (where an error budget that is too small would
  let the screen decide wrongly);
- uniform w3;
plus special cases (w3 = 0 and 2^32 - 1, x below the exp cutoff, tiny and huge
denominators, candidates that are not worse).
"""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sl():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2504_14966_amd.sloanneal as m
    m.load_library()
    return m


def _w3_groups(rng, x, group):
    """w3 for target exponents x by group: 0 boundary, 1 screen edges, 2 uniform."""
    n = x.shape[0]
    e = np.exp(x)
    w_bound = np.floor(e * 2.0**32) + rng.integers(-3, 4, n)
    xl = np.abs(x) * 1.4426950408889634
    tau = xl * 2.0**-16 + 2.0**-10
    s = rng.uniform(0.9, 1.1, n) * np.where(rng.random(n) < 0.5, -1.0, 1.0)
    w_edge = np.floor(e * 2.0 ** (-s * tau) * 2.0**32)
    w_uni = rng.integers(0, 1 << 32, n).astype(np.float64)
    w = np.where(group == 0, w_bound, np.where(group == 1, w_edge, w_uni))
    return np.clip(w, 0, 2.0**32 - 1).astype(np.uint64).astype(np.uint32)


def _inputs_lex(rng, n):
    t_ref = rng.integers(1, 1 << 40, n)
    T = np.exp(rng.uniform(np.log(1e-6), np.log(10.0), n))
    x_target = -np.exp(rng.uniform(np.log(1e-7), np.log(40.0), n))
    delta = np.minimum(np.floor(x_target * t_ref * T), -1).astype(np.int64)
    x = delta / (t_ref.astype(np.float64) * T)
    group = rng.integers(0, 3, n)
    w3 = _w3_groups(rng, x, group)
    return delta, t_ref.astype(np.int64), T, w3, group


def _inputs_ratio(rng, n):
    t = rng.integers(1000, 10**8, n)
    t2 = rng.integers(1000, 10**8, n)
    t_ref = rng.integers(1000, 10**9, n)
    T = np.exp(rng.uniform(np.log(1e-6), np.log(10.0), n))
    x_target = -np.exp(rng.uniform(np.log(1e-7), np.log(40.0), n))
    num = np.minimum(np.floor(x_target * (t.astype(np.float64) * t2) * T / t_ref), -1).astype(np.int64)
    x = (num.astype(np.float64) * t_ref) / ((t.astype(np.float64) * t2) * T)
    group = rng.integers(0, 3, n)
    w3 = _w3_groups(rng, x, group)
    return num, t_ref.astype(np.int64), t.astype(np.int64), t2.astype(np.int64), T, w3, group


def _specials_lex():
    rows = []
    for delta, t_ref, T in ((-1, 10**6, 1.0), (-10**12, 1, 1e-3), (-5, 3, 1e-300), (-5, 10**15, 1e300),
                            (0, 7, 1.0), (12, 7, 0.5), (-(2**62), 1, 1.0), (-1, 1, 1e-20)):
        for w3 in (0, 1, 2**31, 2**32 - 1):
            rows.append((delta, t_ref, T, w3))
    a = np.array(rows, dtype=object)
    return (a[:, 0].astype(np.int64), a[:, 1].astype(np.int64), a[:, 2].astype(np.float64),
            a[:, 3].astype(np.uint64).astype(np.uint32))


def _dev(x, dt):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x)).to(dtype=dt).cuda()


def _run(sl, rule, a, b, T, w3, c=None, d=None):
    import torch
    args = [_dev(a, torch.int64), _dev(b, torch.int64), _dev(T, torch.float64),
            torch.from_numpy(np.ascontiguousarray(w3).view(np.int32)).cuda()]
    kw = {}
    if rule == 1:
        kw = dict(c=_dev(c, torch.int64), d=_dev(d, torch.int64))
    out = sl.sched_accept_check(rule, *args, **kw)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def test_lex_rule_at_the_boundary(sl, orc):
    rng = np.random.default_rng(2024)
    delta, t_ref, T, w3, group = _inputs_lex(rng, 1_200_000)
    sd, st, sT, sw = _specials_lex()
    delta, t_ref, T, w3 = (np.concatenate(p) for p in ((delta, sd), (t_ref, st), (T, sT), (w3, sw)))
    group = np.concatenate([group, np.full(len(sd), 3)])
    got = _run(sl, 0, delta, t_ref, T, w3)
    want = orc.accept_many(0, delta, t_ref, T, w3)
    bad = np.flatnonzero((got & 1) != want)
    assert bad.size == 0, [(int(delta[i]), int(t_ref[i]), float(T[i]), int(w3[i])) for i in bad[:5]]
    screened = (got & 2) != 0
    # the boundary group falls inside the band (where w3 is large enough for a few units to
    # be a small relative step): the double rule decides it
    assert screened[(group == 0) & (w3 >= 1 << 20)].mean() < 0.001
    # at the band edges the screen decides about half, both ways; uniform draws it decides
    g1 = group == 1
    assert 0.2 < screened[g1].mean() < 0.8
    assert (screened & g1 & (want == 1)).any() and (screened & g1 & (want == 0)).any()
    assert screened[group == 2].mean() > 0.99
    # decisions that were not worse, and those of the specials, match too (checked above);
    # every kept / rejected mix is present
    assert 0.05 < want[group < 3].mean() < 0.95


def test_ratio_rule_at_the_boundary(sl, orc):
    rng = np.random.default_rng(77)
    num, t_ref, t, t2, T, w3, group = _inputs_ratio(rng, 1_200_000)
    # specials: not worse, w3 extremes, x below the exp cutoff
    sp = [(0, 5, 100, 100, 1.0, 2**31), (3, 5, 100, 100, 1.0, 0), (-1, 10**9, 10**8, 10**8, 1e-6, 0),
          (-1, 10**9, 10**8, 10**8, 1e-6, 2**32 - 1), (-(10**15), 10**9, 1000, 1000, 1e-6, 1),
          (-1, 1000, 10**8, 10**8, 10.0, 2**32 - 1)]
    sa = np.array(sp, dtype=object)
    num = np.concatenate([num, sa[:, 0].astype(np.int64)])
    t_ref = np.concatenate([t_ref, sa[:, 1].astype(np.int64)])
    t = np.concatenate([t, sa[:, 2].astype(np.int64)])
    t2 = np.concatenate([t2, sa[:, 3].astype(np.int64)])
    T = np.concatenate([T, sa[:, 4].astype(np.float64)])
    w3 = np.concatenate([w3, sa[:, 5].astype(np.uint64).astype(np.uint32)])
    group = np.concatenate([group, np.full(len(sp), 3)])
    got = _run(sl, 1, num, t_ref, T, w3, c=t, d=t2)
    want = orc.accept_many(1, num, t_ref, T, w3, c=t, d=t2)
    bad = np.flatnonzero((got & 1) != want)
    assert bad.size == 0, [(int(num[i]), int(t_ref[i]), int(t[i]), int(t2[i]), float(T[i]), int(w3[i]))
                           for i in bad[:5]]
    screened = (got & 2) != 0
    assert screened[(group == 0) & (w3 >= 1 << 20)].mean() < 0.001
    g1 = group == 1
    assert 0.2 < screened[g1].mean() < 0.8
    assert (screened & g1 & (want == 1)).any() and (screened & g1 & (want == 0)).any()
    assert screened[group == 2].mean() > 0.99
