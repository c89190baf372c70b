"""CPU oracle for the SLO-aware annealing scheduler -- TEST INFRASTRUCTURE ONLY.

Plain single-threaded C (``oracle/*.c``) behind ctypes. Only ``tests/``,
``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may use it;
the GPU library never imports, links or calls it, and it shares no code with the
GPU library.

What it computes and which passage it follows is documented in ``oracle/oracle.h``.
Pins against the paper and the mathematics live in ``tests/test_oracle_*.py``.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRCS = ("replay.c", "rng.c", "anneal.c", "sized.c", "multi.c", "fit.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
CFLAGS = ["-O2", "-std=c99", "-fPIC", "-shared", "-ffp-contract=off", "-fno-fast-math",
          "-Wall", "-Wextra", "-Wno-unused-parameter"]

R_CUR_N, R_CUR_T, R_BEST_N, R_BEST_T, R_BEST_ITER, R_ACCEPTS, R_DIGEST, R_ALLMET = range(8)
TAG_ANNEAL = 0x53414E4E
TAG_FY = 0x46495348


def build(force: bool = True) -> str:
    """Compile the oracle with gcc into oracle/liboracle.so."""
    if force or not os.path.exists(_LIB_PATH):
        tmp = _LIB_PATH + f".tmp{os.getpid()}"
        cmd = ["gcc", *CFLAGS, "-o", tmp, *[os.path.join(_HERE, s) for s in _SRCS], "-lm"]
        subprocess.run(cmd, check=True)
        os.replace(tmp, _LIB_PATH)
    return _LIB_PATH


class _Queue(C.Structure):
    _fields_ = [("n", C.c_int32), ("in_len", C.c_void_p), ("out_len", C.c_void_p),
                ("kind", C.c_void_p), ("thr_us", C.c_void_p)]


class _Model(C.Structure):
    _fields_ = [("max_batch", C.c_int32), ("policy", C.c_int32), ("p0", C.c_int64),
                ("p1", C.c_int64), ("d0", C.c_int64), ("d1", C.c_int64), ("d2", C.c_int64),
                ("t_ref_us", C.c_int64), ("swap_threshold", C.c_uint64)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            build()
        L = C.CDLL(_LIB_PATH)
        vp, i32, i64, u32, u64, dbl = C.c_void_p, C.c_int32, C.c_int64, C.c_uint32, C.c_uint64, C.c_double
        L.orc_replay.argtypes = [vp, vp, vp, vp, vp, vp, vp]
        L.orc_replay.restype = C.c_int
        L.orc_eval_rows.argtypes = [vp, vp, vp, i64, i64, vp]
        L.orc_philox.argtypes = [vp, vp, vp]
        L.orc_det_exp.argtypes = [dbl]
        L.orc_det_exp.restype = dbl
        L.orc_accept.argtypes = [i64, i64, dbl, u32]
        L.orc_accept.restype = C.c_int
        L.orc_fy_perm.argtypes = [u64, i32, u32, vp]
        L.orc_start.argtypes = [vp, vp, vp, vp, vp, vp]
        L.orc_start.restype = C.c_int
        L.orc_swap.argtypes = [vp, i32, i32]
        L.orc_insert.argtypes = [vp, i32, i32]
        L.orc_positions.argtypes = [i32, u32, u32, vp, vp]
        L.orc_anneal_chain.argtypes = [vp, vp, vp, i64, C.c_int, i32, i32, dbl, dbl, u64, vp, vp,
                                       vp, vp]
        L.orc_brute.argtypes = [vp, vp, vp, vp, vp]
        L.orc_brute.restype = i64
        L.orc_solo.argtypes = [vp, vp, i32]
        L.orc_solo.restype = i64
        L.orc_check_starts.argtypes = [vp, i32, i32]
        L.orc_check_starts.restype = C.c_int
        L.orc_max_starts.argtypes = [i32, i32, vp]
        L.orc_replay_batches.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp]
        L.orc_replay_batches.restype = C.c_int
        L.orc_eval_rows_batches.argtypes = [vp, vp, vp, vp, i64, i64, vp]
        L.orc_squeeze.argtypes = [vp, vp, i32, i32, i32]
        L.orc_squeeze.restype = C.c_int
        L.orc_delay.argtypes = [vp, vp, i32, i32, i32]
        L.orc_delay.restype = C.c_int
        L.orc_op3.argtypes = [u32]
        L.orc_op3.restype = C.c_int
        L.orc_anneal_chain_batches.argtypes = [vp, vp, vp, i64, C.c_int, i32, i32, dbl, dbl, u64,
                                               vp, vp, vp, vp, vp, vp]
        L.orc_brute_batches.argtypes = [vp, vp, vp, vp, vp, vp]
        L.orc_brute_batches.restype = i64
        L.orc_better.argtypes = [vp, i64, i64, i64, i64]
        L.orc_better.restype = C.c_int
        L.orc_accept_ratio.argtypes = [i64, i64, i64, i64, dbl, u32]
        L.orc_accept_ratio.restype = C.c_int
        L.orc_accept_many.argtypes = [i32, i64, vp, vp, vp, vp, vp, vp, vp]
        L.orc_accept_many.restype = None
        L.orc_levels.argtypes = [dbl, dbl, dbl]
        L.orc_levels.restype = i32
        L.orc_start_ex.argtypes = [vp, vp, vp, vp, vp, vp, vp]
        L.orc_start_ex.restype = C.c_int
        L.orc_anneal_chain_ex.argtypes = [vp, vp, vp, vp, i64, C.c_int, i32, i32, dbl, dbl, u64, vp, vp, vp, vp]
        L.orc_anneal_chain_batches_ex.argtypes = [vp, vp, vp, vp, i64, C.c_int, i32, i32, dbl, dbl, u64,
                                                  vp, vp, vp, vp, vp, vp]
        L.orc_brute_ex.argtypes = [vp, vp, vp, vp, vp, vp]
        L.orc_brute_ex.restype = i64
        L.orc_assign.argtypes = [vp, i32, vp, vp]
        L.orc_fit_prefill.argtypes = [vp, i64, i64]
        L.orc_fit_prefill.restype = i64
        L.orc_fit_decode.argtypes = [vp, i64, i64, i64]
        L.orc_fit_decode.restype = i64
        L.orc_replay_fit.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp, vp]
        L.orc_replay_fit.restype = C.c_int
        L.orc_start_fit.argtypes = [vp, vp, vp, vp, vp, vp, vp, vp]
        L.orc_start_fit.restype = C.c_int
        L.orc_anneal_chain_fit.argtypes = [vp, vp, vp, vp, vp, i64, C.c_int, i32, i32, dbl, dbl, u64, vp, vp, vp,
                                           vp, vp]
        _lib = L
    return _lib


def _p(a: np.ndarray):
    return a.ctypes.data_as(C.c_void_p)


class _Args:
    """Keeps the contiguous arrays alive while C structs point at them."""

    def __init__(self, queue, model):
        self.in_len = np.ascontiguousarray(queue.in_len, dtype=np.uint16)
        self.out_len = np.ascontiguousarray(queue.out_len, dtype=np.uint16)
        self.kind = np.ascontiguousarray(queue.kind, dtype=np.uint8)
        self.thr = np.ascontiguousarray(queue.thr_us, dtype=np.uint32)
        self.n = int(self.in_len.shape[0])
        self.q = _Queue(self.n, _p(self.in_len).value, _p(self.out_len).value, _p(self.kind).value,
                        _p(self.thr).value)
        self.m = _Model(int(model.max_batch), int(model.policy), int(model.p0), int(model.p1),
                        int(model.d0), int(model.d1), int(model.d2), int(model.t_ref_us),
                        int(model.swap_threshold))
        self.qp = C.byref(self.q)
        self.mp = C.byref(self.m)


def replay(queue, model, perm, detail: bool = False):
    """(n_met, t_sum) of one order, plus per-request (ttft, e2e) when detail is set."""
    a = _Args(queue, model)
    perm = np.ascontiguousarray(perm, dtype=np.uint16)
    nm, ts = C.c_int64(), C.c_int64()
    ttft = np.zeros(a.n, np.int64)
    e2e = np.zeros(a.n, np.int64)
    lib().orc_replay(a.qp, a.mp, _p(perm), C.byref(nm), C.byref(ts), _p(ttft), _p(e2e))
    if detail:
        return nm.value, ts.value, ttft, e2e
    return nm.value, ts.value


def eval_rows(queue, model, perms: np.ndarray, row0: int = 0, rows: int | None = None) -> np.ndarray:
    a = _Args(queue, model)
    perms = np.ascontiguousarray(perms, dtype=np.uint16)
    if rows is None:
        rows = perms.shape[0] - row0
    out = np.zeros((rows, 2), np.int64)
    lib().orc_eval_rows(a.qp, a.mp, _p(perms), row0, rows, _p(out))
    return out


def philox(ctr, key) -> np.ndarray:
    c = np.ascontiguousarray(ctr, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    out = np.zeros(4, np.uint32)
    lib().orc_philox(_p(c), _p(k), _p(out))
    return out


def det_exp(x: float) -> float:
    return lib().orc_det_exp(float(x))


def accept(delta: int, t_ref: int, T: float, w3: int) -> bool:
    return bool(lib().orc_accept(int(delta), int(t_ref), float(T), int(w3)))


def fy_perm(seed: int, n: int, idx: int) -> np.ndarray:
    out = np.zeros(n, np.uint16)
    lib().orc_fy_perm(int(seed), int(n), int(idx), _p(out))
    return out


def fy_perms(seed: int, n: int, rows: int, row0: int = 0) -> np.ndarray:
    return np.stack([fy_perm(seed, n, row0 + k) for k in range(rows)]) if rows else np.zeros((0, n), np.uint16)


def positions(n: int, w1: int, w2: int) -> tuple[int, int]:
    i, j = C.c_int32(), C.c_int32()
    lib().orc_positions(int(n), int(w1), int(w2), C.byref(i), C.byref(j))
    return i.value, j.value


def swap(perm, i, j) -> np.ndarray:
    p = np.array(perm, dtype=np.uint16)
    lib().orc_swap(_p(p), int(i), int(j))
    return p


def insert(perm, i, j) -> np.ndarray:
    p = np.array(perm, dtype=np.uint16)
    lib().orc_insert(_p(p), int(i), int(j))
    return p


def solo(queue, model, r: int) -> int:
    a = _Args(queue, model)
    return lib().orc_solo(a.qp, a.mp, int(r))


OBJ_LEX, OBJ_RATIO = 0, 1


class Search(C.Structure):
    """Search settings: objective (OBJ_LEX attainment then latency, OBJ_RATIO G = n / t),
    proposals per temperature level, early exit when the solo-latency order meets every SLO."""
    _fields_ = [("objective", C.c_int32), ("level_len", C.c_int32), ("early_exit", C.c_int32),
                ("reserved", C.c_int32)]

    def __init__(self, objective=OBJ_LEX, level_len=1, early_exit=0):
        super().__init__(int(objective), int(level_len), int(early_exit), 0)


def _search(search):
    return C.byref(search if search is not None else Search())


def start(queue, model, search: Search | None = None):
    """(start order, t_ref, allmet, start_n, start_t)."""
    a = _Args(queue, model)
    st = np.zeros(a.n, np.uint16)
    t_ref, sn, stt = C.c_int64(), C.c_int64(), C.c_int64()
    allmet = lib().orc_start_ex(a.qp, a.mp, _search(search), _p(st), C.byref(t_ref), C.byref(sn), C.byref(stt))
    return st, t_ref.value, bool(allmet), sn.value, stt.value


def better_key(k1, k2, search: Search | None = None) -> bool:
    return bool(lib().orc_better(_search(search), int(k1[0]), int(k1[1]), int(k2[0]), int(k2[1])))


def accept_ratio(num: int, t_ref: int, t: int, t2: int, T: float, w3: int) -> bool:
    return bool(lib().orc_accept_ratio(int(num), int(t_ref), int(t), int(t2), float(T), int(w3)))


def accept_many(rule: int, a, b, T, w3, c=None, d=None) -> np.ndarray:
    """Acceptance decisions over arrays: rule 0 is accept(a, b, T, w3) (delta, t_ref), rule 1
    accept_ratio(a, b, c, d, T, w3) (num, t_ref, t, t'); uint8 0 / 1 per element."""
    a = np.ascontiguousarray(a, dtype=np.int64)
    k = a.shape[0]
    b = np.ascontiguousarray(b, dtype=np.int64)
    c = np.ascontiguousarray(np.zeros(k) if c is None else c, dtype=np.int64)
    d = np.ascontiguousarray(np.zeros(k) if d is None else d, dtype=np.int64)
    T = np.ascontiguousarray(T, dtype=np.float64)
    w3 = np.ascontiguousarray(w3, dtype=np.uint32)
    assert b.shape == c.shape == d.shape == T.shape == w3.shape == (k,)
    out = np.zeros(k, np.uint8)
    lib().orc_accept_many(int(rule), int(k), _p(a), _p(b), _p(c), _p(d), _p(T), _p(w3), _p(out))
    return out


def levels(T0: float, T_thres: float, tau: float) -> int:
    return int(lib().orc_levels(float(T0), float(T_thres), float(tau)))


def anneal_chain(queue, model, chain: int, iters: int, T0: float, alpha: float, seed: int,
                 start_info=None, trace: bool = False, search: Search | None = None) -> dict:
    """One annealing chain; returns final/best orders, the per-chain record and (optionally) the trace."""
    a = _Args(queue, model)
    if start_info is None:
        start_info = start(queue, model, search)
    st, t_ref, allmet = start_info[0], start_info[1], start_info[2]
    st = np.ascontiguousarray(st, dtype=np.uint16)
    cur = np.zeros(a.n, np.uint16)
    best = np.zeros(a.n, np.uint16)
    rec = np.zeros(8, np.int64)
    tr = np.zeros((iters, 4), np.int64) if trace else None
    lib().orc_anneal_chain_ex(a.qp, a.mp, _search(search), _p(st), int(t_ref), int(allmet), int(chain),
                              int(iters), float(T0), float(alpha), int(seed), _p(cur), _p(best), _p(rec),
                              _p(tr) if trace else None)
    out = dict(cur=cur, best=best, rec=rec)
    if trace:
        out["trace"] = tr
    return out


def brute(queue, model, search: Search | None = None):
    """(best_n, best_t, first optimal order, number of optimal orders) over all n! orders."""
    a = _Args(queue, model)
    if a.n > 10:
        raise ValueError("brute force is limited to n <= 10")
    bn, bt = C.c_int64(), C.c_int64()
    bp = np.zeros(a.n, np.uint16)
    cnt = lib().orc_brute_ex(a.qp, a.mp, _search(search), C.byref(bn), C.byref(bt), _p(bp))
    return bn.value, bt.value, bp, int(cnt)


def better(k1, k2) -> bool:
    """Score order: attainment first, then lower total latency."""
    return k1[0] > k2[0] or (k1[0] == k2[0] and k1[1] < k2[1])


# ---- joint search over order and batch sizes (sized.c) ----

def check_starts(starts, n: int, B: int) -> bool:
    st = np.ascontiguousarray(starts, dtype=np.uint8)
    return bool(lib().orc_check_starts(_p(st), int(n), int(B)))


def max_starts(n: int, B: int) -> np.ndarray:
    st = np.zeros(n, np.uint8)
    lib().orc_max_starts(int(n), int(B), _p(st))
    return st


def replay_batches(queue, model, perm, starts, detail: bool = False):
    """(n_met, t_sum) of one order with explicit batches; (-1, -1) for an invalid row."""
    a = _Args(queue, model)
    perm = np.ascontiguousarray(perm, dtype=np.uint16)
    st = np.ascontiguousarray(starts, dtype=np.uint8)
    nm, ts = C.c_int64(), C.c_int64()
    ttft = np.zeros(a.n, np.int64)
    e2e = np.zeros(a.n, np.int64)
    lib().orc_replay_batches(a.qp, a.mp, _p(perm), _p(st), C.byref(nm), C.byref(ts), _p(ttft), _p(e2e))
    if detail:
        return nm.value, ts.value, ttft, e2e
    return nm.value, ts.value


def eval_rows_batches(queue, model, perms: np.ndarray, starts: np.ndarray) -> np.ndarray:
    a = _Args(queue, model)
    perms = np.ascontiguousarray(perms, dtype=np.uint16)
    st = np.ascontiguousarray(starts, dtype=np.uint8)
    assert perms.shape == st.shape
    out = np.zeros((perms.shape[0], 2), np.int64)
    lib().orc_eval_rows_batches(a.qp, a.mp, _p(perms), _p(st), 0, perms.shape[0], _p(out))
    return out


def squeeze(perm, starts, B: int, i: int):
    """(made, order, starts) after squeezeLastIter at position i."""
    p = np.array(perm, dtype=np.uint16)
    st = np.array(starts, dtype=np.uint8)
    made = lib().orc_squeeze(_p(p), _p(st), int(p.shape[0]), int(B), int(i))
    return bool(made), p, st


def delay(perm, starts, B: int, i: int):
    """(made, order, starts) after delayNextIter at position i."""
    p = np.array(perm, dtype=np.uint16)
    st = np.array(starts, dtype=np.uint8)
    made = lib().orc_delay(_p(p), _p(st), int(p.shape[0]), int(B), int(i))
    return bool(made), p, st


def op3(w0: int) -> int:
    return int(lib().orc_op3(int(w0)))


def anneal_chain_batches(queue, model, chain: int, iters: int, T0: float, alpha: float, seed: int,
                         start_info=None, trace: bool = False, search: Search | None = None) -> dict:
    """One chain of the joint order / batch-size search."""
    a = _Args(queue, model)
    if start_info is None:
        start_info = start(queue, model, search)
    st, t_ref, allmet = start_info[0], start_info[1], start_info[2]
    st = np.ascontiguousarray(st, dtype=np.uint16)
    cur = np.zeros(a.n, np.uint16)
    best = np.zeros(a.n, np.uint16)
    cst = np.zeros(a.n, np.uint8)
    bst = np.zeros(a.n, np.uint8)
    rec = np.zeros(8, np.int64)
    tr = np.zeros((iters, 4), np.int64) if trace else None
    lib().orc_anneal_chain_batches_ex(a.qp, a.mp, _search(search), _p(st), int(t_ref), int(allmet), int(chain),
                                      int(iters), float(T0), float(alpha), int(seed), _p(cur), _p(cst), _p(best),
                                      _p(bst), _p(rec), _p(tr) if trace else None)
    out = dict(cur=cur, cur_starts=cst, best=best, best_starts=bst, rec=rec)
    if trace:
        out["trace"] = tr
    return out


def brute_batches(queue, model):
    """(best_n, best_t, first optimal order, its starts, number of optimal pairs) over every
    order and every batch layout."""
    a = _Args(queue, model)
    if a.n > 8:
        raise ValueError("the joint brute force is limited to n <= 8")
    bn, bt = C.c_int64(), C.c_int64()
    bp = np.zeros(a.n, np.uint16)
    bs = np.zeros(a.n, np.uint8)
    cnt = lib().orc_brute_batches(a.qp, a.mp, C.byref(bn), C.byref(bt), _p(bp), _p(bs))
    return bn.value, bt.value, bp, bs, int(cnt)


# ---- multiple instances (multi.c) ----

def assign(queue, instances: int, capacity) -> np.ndarray:
    """Instance of every request (Scheduling Solution, instance assignment)."""
    a = _Args(queue, _NoModel())
    cap = np.ascontiguousarray(capacity, dtype=np.int64)
    assert cap.shape == (instances,) and 1 <= instances <= 64
    out = np.zeros(a.n, np.int32)
    lib().orc_assign(a.qp, int(instances), _p(cap), _p(out))
    return out


class _NoModel:
    """Model fields for calls that use none of them."""
    max_batch, policy, p0, p1, d0, d1, d2, t_ref_us, swap_threshold = 1, 0, 0, 0, 0, 0, 0, 0, 0


def sub_queue(queue, inst_of, k):
    """The requests of instance k in arrival order, and their ids."""
    from types import SimpleNamespace
    ids = np.flatnonzero(np.asarray(inst_of) == k)
    return SimpleNamespace(in_len=queue.in_len[ids], out_len=queue.out_len[ids], kind=queue.kind[ids],
                           thr_us=queue.thr_us[ids], n=len(ids)), ids


def anneal_instance(queue, model, inst_of, k, chains_per_instance: int, chain: int, iters: int, T0: float,
                    alpha: float, seed: int, search=None) -> dict:
    """Chain `chain` of instance k: the single-queue chain on the instance's requests, drawing
    from Philox chain index k * chains_per_instance + chain."""
    sq, ids = sub_queue(queue, inst_of, k)
    res = anneal_chain(sq, model, k * chains_per_instance + chain, iters, T0, alpha, seed, search=search)
    res["ids"] = ids
    return res


# ---- the fitted latency predictor taken literally (fit.c) ----

KIND_TTFT_TPOT = 3
# Table 2 of the paper (milliseconds), exactly in integer units of 10 ns
TABLE2_10NS = dict(ap=10_000, bp=570_000, cp=1_000, dp=4_367_000, ad=20, bd=27_500, cd=88, dd=1_585_000)


class FitModel(C.Structure):
    _fields_ = [("max_batch", C.c_int32), ("policy", C.c_int32), ("ap", C.c_int64), ("bp", C.c_int64),
                ("cp", C.c_int64), ("dp", C.c_int64), ("ad", C.c_int64), ("bd", C.c_int64), ("cd", C.c_int64),
                ("dd", C.c_int64), ("t_ref", C.c_int64), ("swap_threshold", C.c_uint64)]

    def __init__(self, max_batch, policy=0, ap=0, bp=0, cp=0, dp=0, ad=0, bd=0, cd=0, dd=0, t_ref=0,
                 swap_threshold=1 << 31):
        super().__init__(int(max_batch), int(policy), int(ap), int(bp), int(cp), int(dp), int(ad), int(bd), int(cd),
                         int(dd), int(t_ref), int(swap_threshold))


def _thr2(q, thr2):
    if thr2 is None:
        return None
    a = np.ascontiguousarray(thr2, dtype=np.uint32)
    assert a.shape == (q.n,)
    return a


def fit_prefill(fm: FitModel, b: int, l: int) -> int:
    return int(lib().orc_fit_prefill(C.byref(fm), int(b), int(l)))


def fit_decode(fm: FitModel, b: int, l: int, L: int) -> int:
    return int(lib().orc_fit_decode(C.byref(fm), int(b), int(l), int(L)))


def replay_fit(queue, fm: FitModel, perm, starts=None, thr2=None, detail: bool = False):
    a = _Args(queue, _NoModel())
    perm = np.ascontiguousarray(perm, dtype=np.uint16)
    st = None if starts is None else np.ascontiguousarray(starts, dtype=np.uint8)
    t2 = _thr2(a, thr2)
    nm, ts = C.c_int64(), C.c_int64()
    ttft = np.zeros(a.n, np.int64)
    e2e = np.zeros(a.n, np.int64)
    lib().orc_replay_fit(a.qp, C.byref(fm), _p(perm), _p(st) if st is not None else None,
                         _p(t2) if t2 is not None else None, C.byref(nm), C.byref(ts), _p(ttft), _p(e2e))
    if detail:
        return nm.value, ts.value, ttft, e2e
    return nm.value, ts.value


def start_fit(queue, fm: FitModel, search=None, thr2=None):
    a = _Args(queue, _NoModel())
    t2 = _thr2(a, thr2)
    st = np.zeros(a.n, np.uint16)
    t_ref, sn, stt = C.c_int64(), C.c_int64(), C.c_int64()
    allmet = lib().orc_start_fit(a.qp, C.byref(fm), _search(search), _p(t2) if t2 is not None else None, _p(st),
                                 C.byref(t_ref), C.byref(sn), C.byref(stt))
    return st, t_ref.value, bool(allmet), sn.value, stt.value


def anneal_chain_fit(queue, fm: FitModel, chain: int, iters: int, T0: float, alpha: float, seed: int,
                     search=None, thr2=None, start_info=None) -> dict:
    a = _Args(queue, _NoModel())
    t2 = _thr2(a, thr2)
    if start_info is None:
        start_info = start_fit(queue, fm, search, thr2)
    st, t_ref, allmet = start_info[0], start_info[1], start_info[2]
    st = np.ascontiguousarray(st, dtype=np.uint16)
    cur = np.zeros(a.n, np.uint16)
    best = np.zeros(a.n, np.uint16)
    cst = np.zeros(a.n, np.uint8)
    bst = np.zeros(a.n, np.uint8)
    rec = np.zeros(8, np.int64)
    lib().orc_anneal_chain_fit(a.qp, C.byref(fm), _search(search), _p(t2) if t2 is not None else None, _p(st),
                               int(t_ref), int(allmet), int(chain), int(iters), float(T0), float(alpha), int(seed),
                               _p(cur), _p(cst), _p(best), _p(bst), _p(rec))
    return dict(cur=cur, cur_starts=cst, best=best, best_starts=bst, rec=rec)
