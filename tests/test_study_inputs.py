"""The inputs of the parameter studies and their oracle composition, on the CPU: predicted
output lengths (bounded relative variation; the profiling predictor's class draws),
coefficient variation of one Table 2 parameter, and the invariant that a schedule searched
under the true inputs scores exactly its own chain record."""
import os
import sys

import numpy as np
import pytest

sys.path.insert(0, os.path.dirname(__file__))
from study_oracle import oracle_point  # noqa: E402

from paper_2504_14966_amd.workloads import (OUT_DIST_CHAT, OUT_DIST_CODE, TABLE2_10NS, chat_code_classes,  # noqa: E402
                                            chat_code_queue_10ns, perturbed_fit, perturbed_out_len, sampled_out_len,
                                            two_class_queue)


@pytest.mark.parametrize("v", [0.0, 0.025, 0.05, 0.10])
def test_perturbed_lengths_bounded(v):
    q = two_class_queue(4096, 3)
    p = perturbed_out_len(q.out_len, v, 11)
    L = q.out_len.astype(np.float64)
    assert p.dtype == np.uint16 and p.min() >= 1
    assert np.all(np.abs(p - L) <= v * L + 0.5)
    if v == 0.0:
        assert np.array_equal(p, q.out_len)
    else:
        # u is spread over [-1, 1]: both signs and variations near the bound occur
        r = (p - L) / L
        assert r.min() < -0.8 * v and r.max() > 0.8 * v
    assert np.array_equal(p, perturbed_out_len(q.out_len, v, 11))
    if v > 0:
        assert not np.array_equal(p, perturbed_out_len(q.out_len, v, 12))


def test_class_labels_match_queue():
    # the class draw reproduces two_class_queue's: code requests take the code length law
    n = 2000
    cls = chat_code_classes(n, 5)
    assert int(cls.sum()) == n // 2
    q = two_class_queue(n, 5)
    assert q.out_len[cls == 0].mean() > q.out_len[cls == 1].mean() * 1.3
    q10, thr2 = chat_code_queue_10ns(n, 5)
    assert np.array_equal(q10.kind == 3, cls == 1) and np.array_equal(thr2 > 0, cls == 1)


def test_sampled_lengths_follow_class_law():
    cls = np.repeat(np.array([0, 1], np.uint8), 20000)
    s = sampled_out_len(cls, 4).astype(np.float64)
    assert s.min() >= 1 and s.max() <= 1024
    # the clip at 1 leaves the median of a normal at its mean
    for c, (m, sd) in ((0, OUT_DIST_CODE), (1, OUT_DIST_CHAT)):
        x = s[cls == c]
        assert abs(np.median(x) - m) < 0.03 * m
        # inter-quartile range of a normal: 1.349 SD
        q1, q3 = np.percentile(x, [25, 75])
        assert abs((q3 - q1) / 1.349 - sd) < 0.05 * sd


def test_perturbed_fit():
    assert perturbed_fit(TABLE2_10NS, "a", 0.0) == TABLE2_10NS
    f = perturbed_fit(TABLE2_10NS, "a", 0.05)
    assert f["ap"] == 10_500 and f["ad"] == 21
    assert {k: v for k, v in f.items() if k not in ("ap", "ad")} == \
        {k: v for k, v in TABLE2_10NS.items() if k not in ("ap", "ad")}
    f = perturbed_fit(TABLE2_10NS, "c", -0.1)
    assert f["cp"] == 900 and f["cd"] == 79   # 88 * 0.9 = 79.2
    f = perturbed_fit(TABLE2_10NS, "d", 0.2)
    assert f["dp"] == 5_240_400 and f["dd"] == 1_902_000
    with pytest.raises(ValueError):
        perturbed_fit(TABLE2_10NS, "e", 0.1)


@pytest.mark.parametrize("n,B", [(10, 1), (10, 4)])
def test_unperturbed_point_scores_its_records(orc, n, B):
    q, thr2 = chat_code_queue_10ns(n, 0)
    sc, win, base, iters, recs = oracle_point(orc, q, thr2, TABLE2_10NS, B, range(6), 4.0, 40, 0, T_thres=0.5, tau=0.9)
    assert iters == orc.levels(4.0, 0.5, 0.9) * 40
    assert [tuple(r) for r in sc.tolist()] == recs
    # the winner holds the largest G
    g = [r[0] / r[1] for r in recs]
    assert g[win] == max(g)
    # the baseline is the arrival order in full batches
    f = orc.FitModel(B, 2, **TABLE2_10NS)
    assert base == tuple(orc.replay_fit(q, f, np.arange(n, dtype=np.uint16), orc.max_starts(n, B), thr2))


def test_perturbed_point_differs_only_through_beliefs(orc):
    # a variation of 0 gives the unperturbed point; a large one changes what the chains search
    q, thr2 = chat_code_queue_10ns(10, 0)
    kw = dict(T_thres=0.5, tau=0.9)
    a = oracle_point(orc, q, thr2, TABLE2_10NS, 4, range(4), 4.0, 40, 0, **kw)
    b = oracle_point(orc, q, thr2, TABLE2_10NS, 4, range(4), 4.0, 40, 0,
                     out_len_pred=perturbed_out_len(q.out_len, 0.0, 1), coef_pred=perturbed_fit(TABLE2_10NS, "a", 0.0),
                     **kw)
    assert np.array_equal(a[0], b[0]) and a[1:4] == b[1:4]
    c = oracle_point(orc, q, thr2, TABLE2_10NS, 4, range(4), 4.0, 40, 0,
                     out_len_pred=perturbed_out_len(q.out_len, 0.5, 1), **kw)
    assert c[2] == a[2]  # same baseline
    assert c[4] != a[4]  # the chains saw other lengths
