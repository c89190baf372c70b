"""The paper's parameter studies (Section "Experiments") in model space, on the library.

Each study point runs the paper's scheduler as the experiments configure it -- the ratio
objective G = attainment / mean latency (the objective equation), per-level cooling from T0
down to T_thres = 20 with decay tau = 0.95 and `iter` proposals per level (Algorithm 1),
the early exit, order and batch sizes searched together -- under the latency model and
output lengths the scheduler believes, and scores the schedules it finds under the true
queue and model with sched_eval_fit. Scores are (SLO-met count, sum of end-to-end latencies)
in the fitted model's time unit, so G = n_met / t_sum up to the factor n common to both.

  - T0 / iter study (Fig. 8): believed = true; T0 and iter vary.
  - output-length prediction study (Fig. 9): the scheduler sees predicted output lengths
    (the actual ones varied by a relative amount, or the class-distribution draws of the
    profiling predictor) and is scored on the actual ones.
  - latency-prediction study (Fig. 10): the scheduler sees Table 2 with one parameter
    varied and is scored under Table 2 itself.

The paper runs one chain per schedule. Here every point runs C chains at once: each chain is
one run of the single-chain scheduler (its own Philox stream), so the mean over chains
estimates the expected result of one run, and the winner (the chain the scheduler would
deploy, chosen under the believed model) is reported beside it. The baseline is the arrival
order served in batches of the maximum size, scored under the true model.

Every step runs in the library's kernels; this module only marshals arguments.
"""
from __future__ import annotations

import time
from dataclasses import dataclass, field

import numpy as np

from . import sloanneal as sl
from .workloads import (POLICY_STATIC_SEARCH, TABLE2_10NS, Queue, chat_code_classes, chat_code_queue_10ns,
                        perturbed_fit, perturbed_out_len, sampled_out_len)

T_THRES = 20.0
TAU = 0.95


@dataclass
class StudyPoint:
    label: str
    params: dict
    scores: np.ndarray          # chains x 2 int64: every chain's best schedule under the true model
    winner: int                 # chain chosen by the scheduler (under the model it believes)
    base: tuple                 # (n_met, t_sum) of the arrival order in full batches
    iters: int = 0
    ms: float = 0.0             # wall time of the point (anneal + scoring), host clock
    extra: dict = field(default_factory=dict)

    @property
    def g(self) -> np.ndarray:
        return self.scores[:, 0].astype(np.float64) / self.scores[:, 1].astype(np.float64)

    @property
    def g_base(self) -> float:
        return float(self.base[0]) / float(self.base[1])

    def improvement(self) -> dict:
        """Relative change of G over the baseline: mean over chains, and the winner's."""
        g = self.g
        return dict(mean=float(g.mean() / self.g_base - 1.0), winner=float(g[self.winner] / self.g_base - 1.0))


def fit_model(coef: dict, max_batch: int, policy: int = POLICY_STATIC_SEARCH) -> sl.FitModel:
    return sl.FitModel(max_batch, policy, **coef)


def study_point(label: str, queue: Queue, thr2: np.ndarray, coef: dict, max_batch: int, chains: int, T0: float,
                level_len: int, seed: int, out_len_pred: np.ndarray | None = None, coef_pred: dict | None = None,
                params: dict | None = None, T_thres: float = T_THRES, tau: float = TAU) -> StudyPoint:
    """One schedule search under the believed inputs, scored under the true ones."""
    import torch
    n = queue.n
    q_pred = queue if out_len_pred is None else Queue(queue.in_len, np.ascontiguousarray(out_len_pred, np.uint16),
                                                      queue.kind, queue.thr_us)
    f_true = fit_model(coef, max_batch)
    f_pred = f_true if coef_pred is None else fit_model(coef_pred, max_batch)
    dq_true = sl.DeviceQueue.from_queue(queue)
    dq_pred = dq_true if q_pred is queue else sl.DeviceQueue.from_queue(q_pred)
    t2 = sl.thr_to_device(thr2)
    iters = sl.sched_levels(T0, T_thres, tau) * level_len
    search = sl.Search(sl.OBJ_RATIO, level_len, 1)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ws = sl.sched_anneal_fit(dq_pred, f_pred, chains, iters, T0, tau, seed, tpot_thr=t2, search=search)
    _, _, best = sl.sched_chains(ws, n, chains, perms=True)
    _, best_starts, _ = sl.sched_starts(ws, n, chains)
    _, key = sl.sched_best(ws, n)
    scores = sl.sched_eval_fit(dq_true, f_true, best, best_starts, tpot_thr=t2)
    ident = torch.arange(n, dtype=torch.int16, device=best.device).reshape(1, n)
    base = sl.sched_eval_fit(dq_true, f_true, ident, None, tpot_thr=t2)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3
    b = base.cpu().numpy()[0]
    return StudyPoint(label, dict(params or {}, T0=T0, iter=level_len), scores.cpu().numpy(), int(key[2].item()),
                      (int(b[0]), int(b[1])), iters=iters, ms=ms)


def t0_iter_study(n: int, max_batch: int, T0s=(100.0, 200.0, 300.0, 500.0), level_lens=(50, 100, 200),
                  chains: int = 1024, seed: int = 0, queue_seed: int = 0, coef: dict = TABLE2_10NS, **kw) -> list:
    """Fig. 8 in model space: the chat/code queue of n requests, every (T0, iter) pair."""
    q, thr2 = chat_code_queue_10ns(n, queue_seed)
    return [study_point(f"T0={T0:g} iter={L}", q, thr2, coef, max_batch, chains, T0, L, seed, **kw)
            for T0 in T0s for L in level_lens]


def length_study(n: int, max_batch: int, variations=(0.025, 0.05, 0.10), chains: int = 1024, T0: float = 500.0,
                 level_len: int = 100, seed: int = 0, queue_seed: int = 0, pred_seed: int = 0,
                 coef: dict = TABLE2_10NS, **kw) -> list:
    """Fig. 9 in model space: exact output lengths, the actual ones varied by each relative
    amount, and the class-distribution draws of the profiling predictor."""
    q, thr2 = chat_code_queue_10ns(n, queue_seed)
    preds = [("exact", None, dict(variation=0.0))]
    preds += [(f"variation {v:.1%}", perturbed_out_len(q.out_len, v, pred_seed), dict(variation=v)) for v in variations]
    preds.append(("class distribution", sampled_out_len(chat_code_classes(n, queue_seed), pred_seed),
                  dict(variation=None)))
    return [study_point(lab, q, thr2, coef, max_batch, chains, T0, level_len, seed, out_len_pred=op, params=pp, **kw)
            for lab, op, pp in preds]


def coefficient_study(n: int = 10, max_batch: int = 4, letters: str = "abcd",
                      variations=(-0.2, -0.1, -0.05, 0.05, 0.1, 0.2), chains: int = 1024, T0: float = 500.0,
                      level_len: int = 100, seed: int = 0, queue_seed: int = 0, coef: dict = TABLE2_10NS,
                      **kw) -> list:
    """Fig. 10 in model space: Table 2 itself, then each parameter varied by each amount."""
    q, thr2 = chat_code_queue_10ns(n, queue_seed)
    pts = [study_point("Table 2", q, thr2, coef, max_batch, chains, T0, level_len, seed, params=dict(letter=None),
                       **kw)]
    for a in letters:
        for v in variations:
            pts.append(study_point(f"{a} {v:+.0%}", q, thr2, coef, max_batch, chains, T0, level_len, seed,
                                   coef_pred=perturbed_fit(coef, a, v), params=dict(letter=a, variation=v), **kw))
    return pts
