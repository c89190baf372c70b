"""The parameter studies composed from the oracle: each chain of the paper's scheduler under
the believed queue and model (oracle start and chain), its best schedule replayed under the
true ones, the winner picked by the ratio rule under the believed model (strictly larger
n / t, ties to the lowest chain), and the arrival-order baseline."""
from __future__ import annotations

from fractions import Fraction

import numpy as np

from paper_2504_14966_amd.workloads import POLICY_STATIC_SEARCH, Queue

T_THRES, TAU = 20.0, 0.95


def oracle_point(orc, queue: Queue, thr2, coef: dict, max_batch: int, chains, T0: float, level_len: int,
                 seed: int, out_len_pred=None, coef_pred=None, T_thres: float = T_THRES, tau: float = TAU):
    """(scores chains x 2, winner, base, iters) for the given chain ids."""
    q_pred = queue if out_len_pred is None else Queue(queue.in_len, np.asarray(out_len_pred, np.uint16),
                                                      queue.kind, queue.thr_us)
    f_true = orc.FitModel(max_batch, POLICY_STATIC_SEARCH, **coef)
    f_pred = orc.FitModel(max_batch, POLICY_STATIC_SEARCH, **(coef_pred or coef))
    s = orc.Search(orc.OBJ_RATIO, level_len, 1)
    iters = orc.levels(T0, T_thres, tau) * level_len
    info = orc.start_fit(q_pred, f_pred, s, thr2)
    scores, recs = [], []
    for c in chains:
        w = orc.anneal_chain_fit(q_pred, f_pred, c, iters, T0, tau, seed, search=s, thr2=thr2, start_info=info)
        scores.append(orc.replay_fit(queue, f_true, w["best"], w["best_starts"], thr2))
        recs.append((int(w["rec"][2]), int(w["rec"][3])))
    win = 0
    for k in range(1, len(recs)):
        if Fraction(recs[k][0], recs[k][1]) > Fraction(recs[win][0], recs[win][1]):
            win = k
    base = orc.replay_fit(queue, f_true, np.arange(queue.n, dtype=np.uint16), None, thr2)
    return np.array(scores, np.int64), win, tuple(int(x) for x in base), iters, recs
