"""Seeded synthetic request queues and run settings for the five benchmark workloads.

This module only draws inputs. It holds none of the scheduler's arithmetic (no latency
model evaluation, no objective, no annealing), so both the HIP path and the CPU oracle
can consume what it produces.

Each queue stands in for the paper's evenly mixed, shuffled chat/code request pool
(Section "Experimental setup": ShareGPT-style chat with TTFT/TPOT SLOs and code
completion with an end-to-end SLO, prompt lengths below 2k). The datasets themselves
are not used; only their shape is imitated with lognormal length distributions.

Request attributes follow the problem formulation (Section "Problem Formulation"):
input length l_i, predicted output length l_o, one SLO kind and its threshold in
integer microseconds. Kinds: 0 = TTFT, 1 = TPOT, 2 = end-to-end.
"""
from __future__ import annotations

import hashlib
import math
from dataclasses import dataclass, field

import numpy as np

KIND_TTFT = 0
KIND_TPOT = 1
KIND_E2E = 2

POLICY_STATIC = 0
POLICY_CONTINUOUS = 1
POLICY_STATIC_SEARCH = 2  # static batches whose sizes are searched with the order

# Base SLO thresholds in microseconds, indexed by kind (TTFT, TPOT, E2E).
BASE_THR_SINGLE = (200_000, 50_000, 8_000_000)
BASE_THR_CHAT = BASE_THR_SINGLE
BASE_THR_CODE = (300_000, 75_000, 12_000_000)  # 1.5x: ratio of mean outputs 300/200

# Generation streams: one independent PCG64 stream per purpose.
_S_IN, _S_OUT, _S_KIND, _S_THR, _S_CLASS = 1, 2, 3, 4, 5


@dataclass
class Queue:
    """Structure-of-arrays request queue (length n)."""
    in_len: np.ndarray   # uint16
    out_len: np.ndarray  # uint16, >= 1
    kind: np.ndarray     # uint8 in {0, 1, 2}
    thr_us: np.ndarray   # uint32

    @property
    def n(self) -> int:
        return int(self.in_len.shape[0])

    def sha256(self) -> str:
        h = hashlib.sha256()
        for a in (self.in_len, self.out_len, self.kind, self.thr_us):
            h.update(np.ascontiguousarray(a).tobytes())
        return h.hexdigest()


@dataclass
class Model:
    """Integer-microsecond latency model and admission policy.

    prefill of an admitted group = sum over its requests of (p0 + p1 * l_in);
    one decode step = d0 + d1 * b + d2 * (sum of the active requests' context lengths).
    """
    max_batch: int
    policy: int
    p0: int
    p1: int
    d0: int
    d1: int
    d2: int
    t_ref_us: int = 0
    swap_threshold: int = 1 << 31


@dataclass
class Workload:
    name: str
    queue: Queue
    model: Model
    chains: int = 0
    iters: int = 0
    T0: float = 1.0
    alpha: float = 0.999
    seed: int = 0
    eval_rows: int = 0          # > 0 for the evaluation-only workload
    perm_seed: int = 0
    extra: dict = field(default_factory=dict)


def lognormal_params(mean: float, sd: float) -> tuple[float, float]:
    """(mu, sigma) of the lognormal whose mean and standard deviation are given."""
    s2 = math.log1p((sd / mean) ** 2)
    return math.log(mean) - s2 / 2.0, math.sqrt(s2)


def _rng(seed: int, purpose: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(seed, spawn_key=(purpose,))))


def _lengths(rng, mean, sd, lo, hi, size) -> np.ndarray:
    mu, sigma = lognormal_params(mean, sd)
    x = rng.lognormal(mu, sigma, size=size)
    return np.clip(np.floor(x + 0.5), lo, hi).astype(np.uint16)


def single_class_queue(n: int, seed: int, in_mean=300.0, in_sd=250.0, in_hi=2048) -> Queue:
    """One request class: lognormal input/output lengths, kinds uniform over 3."""
    in_len = _lengths(_rng(seed, _S_IN), in_mean, in_sd, 16, in_hi, n)
    out_len = _lengths(_rng(seed, _S_OUT), 250.0, 200.0, 8, 1024, n)
    kind = _rng(seed, _S_KIND).integers(0, 3, size=n).astype(np.uint8)
    thr = np.asarray(BASE_THR_SINGLE, dtype=np.uint32)[kind]
    return Queue(in_len, out_len, kind, thr.astype(np.uint32))


def two_class_queue(n: int, seed: int, kind_probs=None, thr_jitter=0.0) -> Queue:
    """Evenly mixed code-like and chat-like requests, shuffled.

    Both classes keep the single-class coefficient of variation (input 250/300,
    output 200/250). code: input mean 400, output mean 300; chat: input mean 150,
    output mean 200. With thr_jitter > 0 each threshold is integer-uniform on
    [round((1-j)*base), round((1+j)*base)] of its class.
    """
    if n % 2:
        raise ValueError("two-class queue needs an even n")
    half = n // 2
    cls = np.concatenate([np.zeros(half, np.uint8), np.ones(half, np.uint8)])  # 0 code, 1 chat
    cls = _rng(seed, _S_CLASS).permutation(cls)
    r_in, r_out = _rng(seed, _S_IN), _rng(seed, _S_OUT)
    code_in = _lengths(r_in, 400.0, 400.0 * 250 / 300, 16, 2048, n)
    chat_in = _lengths(r_in, 150.0, 150.0 * 250 / 300, 16, 2048, n)
    code_out = _lengths(r_out, 300.0, 300.0 * 200 / 250, 8, 1024, n)
    chat_out = _lengths(r_out, 200.0, 200.0 * 200 / 250, 8, 1024, n)
    in_len = np.where(cls == 0, code_in, chat_in).astype(np.uint16)
    out_len = np.where(cls == 0, code_out, chat_out).astype(np.uint16)
    rk = _rng(seed, _S_KIND)
    if kind_probs is None:
        kind = rk.integers(0, 3, size=n).astype(np.uint8)
    else:
        kind = rk.choice(3, size=n, p=np.asarray(kind_probs, dtype=np.float64)).astype(np.uint8)
    base = np.where(cls[:, None] == 0, np.asarray(BASE_THR_CODE)[None, :],
                    np.asarray(BASE_THR_CHAT)[None, :])[np.arange(n), kind].astype(np.int64)
    if thr_jitter > 0:
        lo = np.floor((1.0 - thr_jitter) * base + 0.5).astype(np.int64)
        hi = np.floor((1.0 + thr_jitter) * base + 0.5).astype(np.int64)
        thr = _rng(seed, _S_THR).integers(lo, hi + 1)
    else:
        thr = base
    return Queue(in_len, out_len, kind, thr.astype(np.uint32))


def make_queue(n: int, seed: int = 0, in_hi: int = 2048) -> Queue:
    """A small single-class queue for tests (any n >= 1)."""
    return single_class_queue(n, seed, in_hi=in_hi)


def random_queue(rng: np.random.Generator, n: int, max_in=2048, max_out=64, thr_hi=None) -> Queue:
    """Uniformly random small queue for property tests (short outputs keep replays cheap)."""
    in_len = rng.integers(1, max_in + 1, size=n).astype(np.uint16)
    out_len = rng.integers(1, max_out + 1, size=n).astype(np.uint16)
    kind = rng.integers(0, 3, size=n).astype(np.uint8)
    if thr_hi is None:
        thr_hi = 20_000 * n * max_out
    thr = (rng.integers(0, thr_hi, size=n) % 0xFFFFFFFF).astype(np.uint32)  # at most 2^32 - 2
    return Queue(in_len, out_len, kind, thr)


def random_layouts(rng: np.random.Generator, k: int, n: int, B: int) -> np.ndarray:
    """k x n batch-start flags (uint8): batch sizes drawn uniformly from 1..B, last one cut at n."""
    out = np.zeros((k, n), np.uint8)
    for r in range(k):
        p = 0
        while p < n:
            out[r, p] = 1
            p += int(rng.integers(1, B + 1))
    return out


MODEL_A = dict(p0=2000, p1=40, d0=8000, d1=300, d2=2)   # workloads 1, 2, 3, 5
MODEL_B = dict(p0=2000, p1=40, d0=8000, d1=250, d2=1)   # burst workload 4


def workload(idx: int) -> Workload:
    """The five benchmark workloads (1-based index)."""
    if idx == 1:
        return Workload("tiny-n8-b4-static", single_class_queue(8, 0),
                        Model(4, POLICY_STATIC, **MODEL_A), chains=1, iters=2000, T0=1.0, alpha=0.999)
    if idx == 2:
        return Workload("mix-n64-b16-static", two_class_queue(64, 0),
                        Model(16, POLICY_STATIC, **MODEL_A), chains=1024, iters=10000, T0=1.0, alpha=0.999)
    if idx == 3:
        return Workload("mix-n256-b32-continuous", two_class_queue(256, 0, kind_probs=(0.4, 0.3, 0.3),
                                                                   thr_jitter=0.25),
                        Model(32, POLICY_CONTINUOUS, **MODEL_A), chains=2048, iters=20000, T0=1.0, alpha=0.999)
    if idx == 4:
        return Workload("burst-n1024-b64-static", single_class_queue(1024, 0, in_mean=300.0, in_sd=600.0,
                                                                     in_hi=8192),
                        Model(64, POLICY_STATIC, **MODEL_B), chains=4096, iters=5000, T0=2.0, alpha=0.9995)
    if idx == 5:
        return Workload("eval-n128-b16-static", two_class_queue(128, 0),
                        Model(16, POLICY_STATIC, **MODEL_A), eval_rows=1 << 20, perm_seed=0)
    raise ValueError(f"no workload {idx}")


ALL_WORKLOADS = (1, 2, 3, 4, 5)


def search_workload(idx: int) -> Workload:
    """The static annealing workloads (1, 2 or 4) with the batch sizes searched as well:
    same queue, model coefficients, chains, iterations and cooling."""
    W = workload(idx)
    if W.model.policy != POLICY_STATIC or not W.chains:
        raise ValueError(f"workload {idx} is not a static annealing workload")
    m = W.model
    return Workload(W.name.replace("-static", "-search"), W.queue,
                    Model(m.max_batch, POLICY_STATIC_SEARCH, m.p0, m.p1, m.d0, m.d1, m.d2, m.t_ref_us,
                          m.swap_threshold),
                    chains=W.chains, iters=W.iters, T0=W.T0, alpha=W.alpha, seed=W.seed)


def multi_workload() -> Workload:
    """Several serving instances: the two-class 1024-request queue (max batch 16, static)
    spread over 8 instances of 40,000 tokens each by the instance assignment, 512 chains per
    instance (4096 in all) x 2000 proposals, T0 1.0, alpha 0.999."""
    W = Workload("multi-8x-n1024-b16-static", two_class_queue(1024, 0), Model(16, POLICY_STATIC, **MODEL_A),
                 chains=512, iters=2000, T0=1.0, alpha=0.999)
    W.extra = dict(instances=8, capacity=[40_000] * 8)
    return W


# Table 2 of the paper (milliseconds) in integer units of 10 ns
TABLE2_10NS = dict(ap=10_000, bp=570_000, cp=1_000, dp=4_367_000, ad=20, bd=27_500, cd=88, dd=1_585_000)


def chat_code_queue_10ns(n: int, seed: int):
    """The two-class queue for the fitted model: code requests keep an end-to-end SLO, chat
    requests take the paper's chat SLO (TTFT and TPOT together); thresholds in units of
    10 ns. Code: e2e 30 s; chat: TTFT 10 s and TPOT 50 ms (the paper's SLO settings).
    Returns the queue and the per-request TPOT thresholds (0 for code requests)."""
    q = two_class_queue(n, seed)
    # the class labels two_class_queue drew (same stream): 0 code, 1 chat
    cls = _rng(seed, _S_CLASS).permutation(np.concatenate([np.zeros(n // 2, np.uint8), np.ones(n // 2, np.uint8)]))
    kind = np.where(cls == 0, 2, 3).astype(np.uint8)
    thr = np.where(cls == 0, 3_000_000_000, 1_000_000_000).astype(np.uint32)
    thr2 = np.where(cls == 0, 0, 5_000_000).astype(np.uint32)
    return Queue(q.in_len, q.out_len, kind, thr), thr2


# ---- inputs of the parameter studies (Experiments) ----

_S_PRED, _S_SAMPLE = 6, 7

# Output-length distributions of the two classes as two_class_queue draws them: (mean, SD)
OUT_DIST_CODE = (300.0, 300.0 * 200 / 250)
OUT_DIST_CHAT = (200.0, 200.0 * 200 / 250)

# The scenarios of the T0 / iter study and of the output-length study: (requests, max batch)
STUDY_SCENARIOS = ((10, 1), (20, 2), (40, 4))


def chat_code_classes(n: int, seed: int) -> np.ndarray:
    """Class of every request of two_class_queue(n, seed) (same stream): 0 code, 1 chat."""
    return _rng(seed, _S_CLASS).permutation(np.concatenate([np.zeros(n // 2, np.uint8), np.ones(n // 2, np.uint8)]))


def perturbed_out_len(out_len: np.ndarray, variation: float, seed: int) -> np.ndarray:
    """Predicted output lengths within a relative variation of the actual ones (the Impact of
    Output Length Prediction study: actual lengths varied by 2.5, 5 or 10 %): l (1 + v u)
    with u uniform on [-1, 1], rounded to the nearest integer, kept in [1, 65535]."""
    u = _rng(seed, _S_PRED).uniform(-1.0, 1.0, size=out_len.shape[0])
    x = out_len.astype(np.float64) * (1.0 + variation * u)
    return np.clip(np.floor(x + 0.5), 1, 65535).astype(np.uint16)


def sampled_out_len(cls: np.ndarray, seed: int) -> np.ndarray:
    """The profiling-based predictor of the paper's setup: for every request a random integer
    from the normal distribution with its class's output-length mean and SD, rounded to the
    nearest integer and kept in [1, 1024] (the range two_class_queue draws from)."""
    r = _rng(seed, _S_SAMPLE)
    mean = np.where(cls == 0, OUT_DIST_CODE[0], OUT_DIST_CHAT[0])
    sd = np.where(cls == 0, OUT_DIST_CODE[1], OUT_DIST_CHAT[1])
    x = r.normal(mean, sd)
    return np.clip(np.floor(x + 0.5), 1, 1024).astype(np.uint16)


def perturbed_fit(coef: dict, letter: str, variation: float) -> dict:
    """Latency-predictor coefficients with one parameter of Table 2 varied (the Impact of
    Latency Prediction study): the prefill and decode coefficients named by `letter`
    ('a' alpha: b l, 'b' beta: b, 'c' gamma: l, 'd' delta: constant) scaled by
    (1 + variation) and rounded to the nearest integer; every other coefficient unchanged."""
    if letter not in "abcd" or len(letter) != 1:
        raise ValueError("letter is one of a, b, c, d")
    out = dict(coef)
    for k in (letter + "p", letter + "d"):
        out[k] = int(math.floor(coef[k] * (1.0 + variation) + 0.5))
    return out
