"""GPU parity of the parameter studies in model space against their oracle composition,
bit for bit: every chain's best schedule scored under the true queue and model, the chain
the scheduler picks under the model it believes, and the arrival-order baseline -- for the
T0 / iter study, the output-length prediction study and the coefficient study."""
import os
import sys

import numpy as np
import pytest

sys.path.insert(0, os.path.dirname(__file__))
from study_oracle import oracle_point  # noqa: E402

from paper_2504_14966_amd.workloads import (TABLE2_10NS, chat_code_classes, chat_code_queue_10ns,  # noqa: E402
                                            perturbed_fit, perturbed_out_len, sampled_out_len)

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def st():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2504_14966_amd.sloanneal as sl
    sl.load_library()
    import paper_2504_14966_amd.studies as m
    return m


def _same(p, want):
    sc, win, base, iters, _ = want
    assert p.iters == iters, p.label
    assert p.scores.tolist() == sc.tolist(), p.label
    assert p.winner == win and p.base == base, p.label


LOW = dict(T_thres=0.5, tau=0.9)


@pytest.mark.parametrize("n,B", [(10, 1), (10, 4), (20, 2)])
def test_t0_iter_study(st, orc, n, B):
    pts = st.t0_iter_study(n, B, T0s=(2.0, 4.0), level_lens=(10, 40), chains=12, seed=3, **LOW)
    q, thr2 = chat_code_queue_10ns(n, 0)
    assert len(pts) == 4
    for p in pts:
        _same(p, oracle_point(orc, q, thr2, TABLE2_10NS, B, range(12), p.params["T0"], p.params["iter"], 3, **LOW))


def test_t0_iter_study_paper_schedule(st, orc):
    # T0 = 500 cooled by 0.95 to 20: 63 levels of `iter` proposals
    pts = st.t0_iter_study(10, 1, T0s=(500.0,), level_lens=(20,), chains=6, seed=1)
    q, thr2 = chat_code_queue_10ns(10, 0)
    assert pts[0].iters == 63 * 20
    _same(pts[0], oracle_point(orc, q, thr2, TABLE2_10NS, 1, range(6), 500.0, 20, 1))


def test_length_study(st, orc):
    pts = st.length_study(10, 4, variations=(0.05, 0.25), chains=8, T0=4.0, level_len=30, seed=2, **LOW)
    q, thr2 = chat_code_queue_10ns(10, 0)
    preds = [None, perturbed_out_len(q.out_len, 0.05, 0), perturbed_out_len(q.out_len, 0.25, 0),
             sampled_out_len(chat_code_classes(10, 0), 0)]
    assert [p.label for p in pts][0] == "exact" and len(pts) == 4
    for p, op in zip(pts, preds):
        _same(p, oracle_point(orc, q, thr2, TABLE2_10NS, 4, range(8), 4.0, 30, 2, out_len_pred=op, **LOW))
    # under exact lengths each chain scores its own record
    assert pts[0].improvement()["winner"] >= pts[0].improvement()["mean"]


def test_coefficient_study(st, orc):
    pts = st.coefficient_study(10, 4, letters="ad", variations=(-0.2, 0.1), chains=8, T0=4.0, level_len=30, seed=5,
                               **LOW)
    q, thr2 = chat_code_queue_10ns(10, 0)
    want = [None] + [perturbed_fit(TABLE2_10NS, a, v) for a in "ad" for v in (-0.2, 0.1)]
    assert len(pts) == 5
    for p, cp in zip(pts, want):
        _same(p, oracle_point(orc, q, thr2, TABLE2_10NS, 4, range(8), 4.0, 30, 5, coef_pred=cp, **LOW))
