"""ctypes binding of libsloanneal.so (C-ABI in include/sloanneal.h).

Argument marshalling only: every step of the scheduler runs in the library's HIP
kernels. torch supplies device memory and the stream. There is no CPU fallback: if
the library or a GPU is missing, every call raises.
"""
from __future__ import annotations

import ctypes as C
import os
from dataclasses import dataclass

import numpy as np
import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libsloanneal.so")

SCHED_OK, SCHED_EINVAL, SCHED_ENOSPC, SCHED_ERANGE, SCHED_EHIP = 0, -1, -2, -3, -4
EXPORTS = ("sched_eval", "sched_eval_batches", "sched_ws_bytes", "sched_anneal", "sched_anneal_ex", "sched_levels",
           "sched_best", "sched_chains", "sched_start_info", "sched_starts", "sched_gen_perms", "sched_assign",
           "sched_ws_bytes_multi", "sched_anneal_multi", "sched_multi_instance_ws", "sched_multi_best",
           "sched_eval_fit", "sched_anneal_fit", "sched_accept_check", "sched_anneal_noalloc", "sched_status",
           "sched_strerror")
# width flags of the device checks (sched_status word 1)
FLAG_NARROW_PREFILL, FLAG_LIST_SCHED, FLAG_NARROW_TIME, FLAG_WINDOWS = 1, 2, 4, 8
FLAG_STATIC_NARROW, FLAG_TIME32, FLAG_FIT_WINDOWS, FLAG_FIT_MEMBER32 = 16, 32, 64, 128
FLAG_INST64, FLAG_INST192 = 256, 512
KIND_TTFT_TPOT = 3
POLICY_STATIC, POLICY_CONTINUOUS, POLICY_STATIC_SEARCH = 0, 1, 2
OBJ_LEX, OBJ_RATIO = 0, 1


class SchedError(RuntimeError):
    def __init__(self, code: int, msg: str):
        super().__init__(f"{msg} (code {code})")
        self.code = code


class _Queue(C.Structure):
    _fields_ = [("n", C.c_int32), ("in_len", C.c_void_p), ("out_len", C.c_void_p), ("kind", C.c_void_p),
                ("thr_us", C.c_void_p)]


class Search(C.Structure):
    """Search settings (sched_search_t): objective OBJ_LEX or OBJ_RATIO, proposals per
    temperature level, early exit when the solo-latency order meets every SLO."""
    _fields_ = [("objective", C.c_int32), ("level_len", C.c_int32), ("early_exit", C.c_int32),
                ("reserved", C.c_int32)]

    def __init__(self, objective=OBJ_LEX, level_len=1, early_exit=0):
        super().__init__(int(objective), int(level_len), int(early_exit), 0)


class _Model(C.Structure):
    _fields_ = [("max_batch", C.c_int32), ("policy", C.c_int32), ("p0", C.c_int64), ("p1", C.c_int64),
                ("d0", C.c_int64), ("d1", C.c_int64), ("d2", C.c_int64), ("t_ref_us", C.c_int64),
                ("swap_threshold", C.c_uint64)]


_lib = None


def load_library(path: str = LIB_PATH):
    """dlopen the library and declare its signatures (no GPU needed)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise RuntimeError(f"libsloanneal.so is not built ({path}); run __graft_entry__.build()")
    L = C.CDLL(path)
    vp, i32, i64, u64, dbl, sz = C.c_void_p, C.c_int32, C.c_int64, C.c_uint64, C.c_double, C.c_size_t
    L.sched_eval.argtypes = [vp, vp, vp, i64, vp, vp, vp]
    L.sched_eval.restype = C.c_int
    L.sched_eval_batches.argtypes = [vp, vp, vp, vp, i64, vp, vp, vp]
    L.sched_eval_batches.restype = C.c_int
    L.sched_starts.argtypes = [vp, vp, vp, vp, vp]
    L.sched_starts.restype = C.c_int
    L.sched_ws_bytes.argtypes = [i32, i32]
    L.sched_ws_bytes.restype = sz
    L.sched_anneal.argtypes = [vp, vp, i32, i32, dbl, dbl, u64, vp, sz, vp]
    L.sched_anneal.restype = C.c_int
    L.sched_anneal_ex.argtypes = [vp, vp, vp, i32, i32, dbl, dbl, u64, vp, sz, vp]
    L.sched_anneal_ex.restype = C.c_int
    L.sched_levels.argtypes = [dbl, dbl, dbl]
    L.sched_levels.restype = i32
    L.sched_assign.argtypes = [vp, i32, vp, vp, vp]
    L.sched_assign.restype = C.c_int
    L.sched_ws_bytes_multi.argtypes = [i32, i32, i32]
    L.sched_ws_bytes_multi.restype = sz
    L.sched_anneal_multi.argtypes = [vp, vp, vp, vp, i32, i32, i32, dbl, dbl, u64, vp, sz, vp]
    L.sched_anneal_multi.restype = C.c_int
    L.sched_multi_instance_ws.argtypes = [vp, i32, i32, i32, i32]
    L.sched_multi_instance_ws.restype = vp
    L.sched_multi_best.argtypes = [vp, i32, vp, vp, vp, vp]
    L.sched_multi_best.restype = C.c_int
    L.sched_eval_fit.argtypes = [vp, vp, vp, vp, vp, i64, vp, vp, vp]
    L.sched_eval_fit.restype = C.c_int
    L.sched_anneal_fit.argtypes = [vp, vp, vp, vp, i32, i32, dbl, dbl, u64, vp, sz, vp]
    L.sched_anneal_fit.restype = C.c_int
    L.sched_best.argtypes = [vp, vp, vp, vp]
    L.sched_best.restype = C.c_int
    L.sched_chains.argtypes = [vp, vp, vp, vp, vp]
    L.sched_chains.restype = C.c_int
    L.sched_start_info.argtypes = [vp, vp, vp, vp]
    L.sched_start_info.restype = C.c_int
    L.sched_gen_perms.argtypes = [u64, i32, i64, i64, vp, vp]
    L.sched_gen_perms.restype = C.c_int
    L.sched_anneal_noalloc.argtypes = [vp, vp, i32, i32, dbl, dbl, u64, vp, vp, vp]
    L.sched_anneal_noalloc.restype = C.c_int
    L.sched_accept_check.argtypes = [i32, i64, vp, vp, vp, vp, vp, vp, vp, vp]
    L.sched_accept_check.restype = C.c_int
    L.sched_status.argtypes = [vp, vp, vp]
    L.sched_status.restype = C.c_int
    L.sched_strerror.argtypes = [C.c_int]
    L.sched_strerror.restype = C.c_char_p
    _lib = L
    return L


def _check(rc: int):
    if rc != SCHED_OK:
        raise SchedError(rc, load_library().sched_strerror(rc).decode())


def _stream(stream) -> C.c_void_p:
    s = stream if stream is not None else torch.cuda.current_stream()
    return C.c_void_p(s.cuda_stream)


def _ptr(t: torch.Tensor | None):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("sloanneal takes device tensors")
    if not t.is_contiguous():
        raise ValueError("sloanneal takes contiguous tensors")
    return C.c_void_p(t.data_ptr())


@dataclass
class DeviceQueue:
    """A request queue resident in device memory (structure of arrays)."""
    in_len: torch.Tensor   # int16 bits of uint16
    out_len: torch.Tensor
    kind: torch.Tensor     # uint8
    thr_us: torch.Tensor   # int32 bits of uint32

    @property
    def n(self) -> int:
        return int(self.in_len.shape[0])

    @classmethod
    def from_queue(cls, q, device="cuda") -> "DeviceQueue":
        def dev(a, np_dt, t_dt):
            return torch.from_numpy(np.ascontiguousarray(a, dtype=np_dt).view(t_dt)).to(device)
        return cls(dev(q.in_len, np.uint16, np.int16), dev(q.out_len, np.uint16, np.int16),
                   dev(q.kind, np.uint8, np.uint8), dev(q.thr_us, np.uint32, np.int32))

    def c(self) -> _Queue:
        return _Queue(self.n, self.in_len.data_ptr(), self.out_len.data_ptr(), self.kind.data_ptr(),
                      self.thr_us.data_ptr())


def _model(m) -> _Model:
    return _Model(int(m.max_batch), int(m.policy), int(m.p0), int(m.p1), int(m.d0), int(m.d1), int(m.d2),
                  int(m.t_ref_us), int(m.swap_threshold))


def perms_to_device(perms: np.ndarray, device="cuda") -> torch.Tensor:
    """k x n orders as an int16 device tensor holding the uint16 bits."""
    return torch.from_numpy(np.ascontiguousarray(perms, dtype=np.uint16).view(np.int16)).to(device)


def sched_eval(dq: DeviceQueue, model, perms: torch.Tensor, out: torch.Tensor | None = None,
               detail: bool | torch.Tensor = False, stream=None):
    """(n_met, t_sum) per row of perms (k x n, int16/uint16 bits); optionally per-request (ttft, e2e)."""
    L = load_library()
    k = int(perms.shape[0]) if perms.dim() == 2 else 0
    if perms.dim() != 2 or int(perms.shape[1]) != dq.n:
        raise ValueError("perms must be k x n")
    if out is None:
        out = torch.empty((k, 2), dtype=torch.int64, device=perms.device)
    det = None
    if isinstance(detail, torch.Tensor):
        det = detail
    elif detail:
        det = torch.zeros((k, dq.n, 2), dtype=torch.int64, device=perms.device)
    q, m = dq.c(), _model(model)
    _check(L.sched_eval(C.byref(q), C.byref(m), _ptr(perms), k, _ptr(out), _ptr(det), _stream(stream)))
    return (out, det) if det is not None else out


def starts_to_device(starts: np.ndarray, device="cuda") -> torch.Tensor:
    """k x n batch-start flags as a uint8 device tensor."""
    return torch.from_numpy(np.ascontiguousarray(starts, dtype=np.uint8)).to(device)


def sched_eval_batches(dq: DeviceQueue, model, perms: torch.Tensor, starts: torch.Tensor,
                       out: torch.Tensor | None = None, detail: bool | torch.Tensor = False, stream=None):
    """(n_met, t_sum) per (order, layout) row: perms k x n (uint16 bits), starts k x n uint8."""
    L = load_library()
    if perms.dim() != 2 or int(perms.shape[1]) != dq.n or tuple(starts.shape) != tuple(perms.shape):
        raise ValueError("perms and starts must both be k x n")
    if starts.dtype != torch.uint8:
        raise ValueError("starts must be uint8")
    k = int(perms.shape[0])
    if out is None:
        out = torch.empty((k, 2), dtype=torch.int64, device=perms.device)
    det = None
    if isinstance(detail, torch.Tensor):
        det = detail
    elif detail:
        det = torch.zeros((k, dq.n, 2), dtype=torch.int64, device=perms.device)
    q, m = dq.c(), _model(model)
    _check(L.sched_eval_batches(C.byref(q), C.byref(m), _ptr(perms), _ptr(starts), k, _ptr(out), _ptr(det),
                                _stream(stream)))
    return (out, det) if det is not None else out


def ws_bytes(n: int, chains: int) -> int:
    return int(load_library().sched_ws_bytes(int(n), int(chains)))


def alloc_ws(n: int, chains: int, device="cuda") -> torch.Tensor:
    nb = ws_bytes(n, chains)
    if nb == 0:
        raise ValueError("bad workspace size request")
    return torch.empty(nb, dtype=torch.uint8, device=device)


def sched_anneal(dq: DeviceQueue, model, chains: int, iters: int, T0: float, alpha: float, seed: int,
                 ws: torch.Tensor | None = None, stream=None, search: Search | None = None) -> torch.Tensor:
    """Run the chains; with `search`, sched_anneal_ex (objective, per-level cooling, early exit)."""
    L = load_library()
    if ws is None:
        ws = alloc_ws(dq.n, chains)
    q, m = dq.c(), _model(model)
    if search is None:
        _check(L.sched_anneal(C.byref(q), C.byref(m), int(chains), int(iters), float(T0), float(alpha),
                              int(seed) & (2**64 - 1), _ptr(ws), int(ws.numel()), _stream(stream)))
    else:
        _check(L.sched_anneal_ex(C.byref(q), C.byref(m), C.byref(search), int(chains), int(iters), float(T0),
                                 float(alpha), int(seed) & (2**64 - 1), _ptr(ws), int(ws.numel()), _stream(stream)))
    return ws


def sched_anneal_noalloc(dq: DeviceQueue, model, chains: int, iters: int, T0: float, alpha: float, seed: int,
                         perm_out: torch.Tensor | None = None, key_out: torch.Tensor | None = None, stream=None):
    """sched_anneal + sched_best in the library's fixed device scratch (the C call allocates
    nothing; outputs are allocated here unless given): (best order n int16 bits, key 3 int64)."""
    dev = dq.in_len.device
    perm = perm_out if perm_out is not None else torch.empty(dq.n, dtype=torch.int16, device=dev)
    key = key_out if key_out is not None else torch.empty(3, dtype=torch.int64, device=dev)
    q, m = dq.c(), _model(model)
    _check(load_library().sched_anneal_noalloc(C.byref(q), C.byref(m), int(chains), int(iters), float(T0),
                                               float(alpha), int(seed) & (2**64 - 1), _ptr(perm), _ptr(key),
                                               _stream(stream)))
    return perm, key


def sched_levels(T0: float, T_thres: float, tau: float) -> int:
    """Temperature levels of Algorithm 1 (T0 cooled by tau until below T_thres)."""
    v = int(load_library().sched_levels(float(T0), float(T_thres), float(tau)))
    if v < 0:
        raise SchedError(v, load_library().sched_strerror(v).decode())
    return v


def sched_best(ws: torch.Tensor, n: int, stream=None):
    perm = torch.empty(n, dtype=torch.int16, device=ws.device)
    key = torch.empty(3, dtype=torch.int64, device=ws.device)
    _check(load_library().sched_best(_ptr(ws), _ptr(perm), _ptr(key), _stream(stream)))
    return perm, key


def sched_status(ws: torch.Tensor, stream=None) -> torch.Tensor:
    """The device checks' verdict of the last annealing call on ws (a single-queue, several-
    instance or instance workspace): 3 int64 on the device (status, width flags, selected
    kernel among the call's candidates or -1)."""
    out = torch.empty(3, dtype=torch.int64, device=ws.device)
    _check(load_library().sched_status(_ptr(ws), _ptr(out), _stream(stream)))
    return out


def sched_chains(ws: torch.Tensor, n: int, chains: int, perms: bool = False, stream=None):
    rec = torch.empty((chains, 8), dtype=torch.int64, device=ws.device)
    cur = best = None
    if perms:
        cur = torch.empty((chains, n), dtype=torch.int16, device=ws.device)
        best = torch.empty((chains, n), dtype=torch.int16, device=ws.device)
    _check(load_library().sched_chains(_ptr(ws), _ptr(rec), _ptr(cur), _ptr(best), _stream(stream)))
    return (rec, cur, best) if perms else rec


def sched_start_info(ws: torch.Tensor, n: int, stream=None):
    start = torch.empty(n, dtype=torch.int16, device=ws.device)
    info = torch.empty(4, dtype=torch.int64, device=ws.device)
    _check(load_library().sched_start_info(_ptr(ws), _ptr(start), _ptr(info), _stream(stream)))
    return start, info


def sched_starts(ws: torch.Tensor, n: int, chains: int, stream=None):
    """Batch layouts after a batch-size search: (cur chains x n, best chains x n, winner n), uint8."""
    cur = torch.empty((chains, n), dtype=torch.uint8, device=ws.device)
    best = torch.empty((chains, n), dtype=torch.uint8, device=ws.device)
    win = torch.empty(n, dtype=torch.uint8, device=ws.device)
    _check(load_library().sched_starts(_ptr(ws), _ptr(cur), _ptr(best), _ptr(win), _stream(stream)))
    return cur, best, win


def sched_gen_perms(seed: int, n: int, k: int, row0: int = 0, out: torch.Tensor | None = None, stream=None,
                    device="cuda") -> torch.Tensor:
    if out is None:
        out = torch.empty((k, n), dtype=torch.int16, device=device)
    _check(load_library().sched_gen_perms(int(seed) & (2**64 - 1), int(n), int(row0), int(k), _ptr(out),
                                          _stream(stream)))
    return out


def as_u16(t: torch.Tensor) -> np.ndarray:
    """Host numpy uint16 view of an int16 device tensor."""
    return t.cpu().numpy().view(np.uint16)


# ---- several serving instances ----

def sched_assign(dq: DeviceQueue, capacity: torch.Tensor, stream=None) -> torch.Tensor:
    """Instance of every request (capacity: int64 device tensor, tokens per instance)."""
    out = torch.empty(dq.n, dtype=torch.int32, device=capacity.device)
    q = dq.c()
    _check(load_library().sched_assign(C.byref(q), int(capacity.numel()), _ptr(capacity), _ptr(out), _stream(stream)))
    return out


class MultiWorkspace:
    """A sched_anneal_multi workspace and the single-queue views of its instances."""

    def __init__(self, n: int, instances: int, chains: int, device="cuda"):
        nb = int(load_library().sched_ws_bytes_multi(int(n), int(instances), int(chains)))
        if nb == 0:
            raise ValueError("bad multi-instance workspace size request")
        self.n, self.instances, self.chains = int(n), int(instances), int(chains)
        self.buf = torch.empty(nb, dtype=torch.uint8, device=device)

    def instance(self, k: int) -> torch.Tensor:
        """Instance k's workspace, as a view usable with sched_best / sched_chains / sched_start_info."""
        p = load_library().sched_multi_instance_ws(_ptr(self.buf), self.n, self.instances, self.chains, int(k))
        if not p:
            raise ValueError("bad instance")
        off = int(p) - self.buf.data_ptr()
        return self.buf[off:]


def sched_anneal_multi(dq: DeviceQueue, model, inst_of: torch.Tensor, instances: int, chains: int, iters: int,
                       T0: float, alpha: float, seed: int, search: Search | None = None,
                       mws: MultiWorkspace | None = None, stream=None) -> MultiWorkspace:
    L = load_library()
    if mws is None:
        mws = MultiWorkspace(dq.n, instances, chains, device=inst_of.device)
    q, m = dq.c(), _model(model)
    _check(L.sched_anneal_multi(C.byref(q), C.byref(m), C.byref(search) if search is not None else None,
                                _ptr(inst_of), int(instances), int(chains), int(iters), float(T0), float(alpha),
                                int(seed) & (2**64 - 1), _ptr(mws.buf), int(mws.buf.numel()), _stream(stream)))
    return mws


def sched_multi_status(mws: MultiWorkspace, stream=None) -> torch.Tensor:
    return sched_status(mws.buf, stream)


def sched_multi_best(mws: MultiWorkspace, stream=None):
    """(orders n uint16 bits: each instance's best order as global ids, instance after
    instance; keys instances x 3; counts instances)."""
    dev = mws.buf.device
    orders = torch.empty(mws.n, dtype=torch.int16, device=dev)
    keys = torch.empty((mws.instances, 3), dtype=torch.int64, device=dev)
    counts = torch.empty(mws.instances, dtype=torch.int32, device=dev)
    _check(load_library().sched_multi_best(_ptr(mws.buf), mws.instances, _ptr(orders), _ptr(keys), _ptr(counts),
                                           _stream(stream)))
    return orders, keys, counts


# ---- the fitted latency model ----

class FitModel(C.Structure):
    """sched_fit_model_t: per-request prefill ap*b*l + bp*b + cp*l + dp and per-token decode
    ad*b*l + bd*b + cd*l + dd in one integer time unit (Table 2 in units of 10 ns: TABLE2_10NS)."""
    _fields_ = [("max_batch", C.c_int32), ("policy", C.c_int32), ("ap", C.c_int64), ("bp", C.c_int64),
                ("cp", C.c_int64), ("dp", C.c_int64), ("ad", C.c_int64), ("bd", C.c_int64), ("cd", C.c_int64),
                ("dd", C.c_int64), ("t_ref", C.c_int64), ("swap_threshold", C.c_uint64)]

    def __init__(self, max_batch, policy=0, ap=0, bp=0, cp=0, dp=0, ad=0, bd=0, cd=0, dd=0, t_ref=0,
                 swap_threshold=1 << 31):
        super().__init__(int(max_batch), int(policy), int(ap), int(bp), int(cp), int(dp), int(ad), int(bd), int(cd),
                         int(dd), int(t_ref), int(swap_threshold))


TABLE2_10NS = dict(ap=10_000, bp=570_000, cp=1_000, dp=4_367_000, ad=20, bd=27_500, cd=88, dd=1_585_000)


def thr_to_device(thr: np.ndarray, device="cuda") -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(thr, dtype=np.uint32).view(np.int32)).to(device)


def sched_eval_fit(dq: DeviceQueue, fit: FitModel, perms: torch.Tensor, starts: torch.Tensor | None = None,
                   tpot_thr: torch.Tensor | None = None, detail: bool = False, stream=None):
    L = load_library()
    k = int(perms.shape[0])
    if perms.dim() != 2 or int(perms.shape[1]) != dq.n:
        raise ValueError("perms must be k x n")
    if starts is not None and (tuple(starts.shape) != tuple(perms.shape) or starts.dtype != torch.uint8):
        raise ValueError("starts must be k x n uint8")
    out = torch.empty((k, 2), dtype=torch.int64, device=perms.device)
    det = torch.zeros((k, dq.n, 2), dtype=torch.int64, device=perms.device) if detail else None
    q = dq.c()
    _check(L.sched_eval_fit(C.byref(q), C.byref(fit), _ptr(tpot_thr), _ptr(perms), _ptr(starts), k, _ptr(out),
                            _ptr(det), _stream(stream)))
    return (out, det) if detail else out


def sched_anneal_fit(dq: DeviceQueue, fit: FitModel, chains: int, iters: int, T0: float, alpha: float, seed: int,
                     tpot_thr: torch.Tensor | None = None, search: Search | None = None,
                     ws: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    L = load_library()
    if ws is None:
        ws = alloc_ws(dq.n, chains)
    q = dq.c()
    _check(L.sched_anneal_fit(C.byref(q), C.byref(fit), _ptr(tpot_thr), C.byref(search) if search is not None else None,
                              int(chains), int(iters), float(T0), float(alpha), int(seed) & (2**64 - 1), _ptr(ws),
                              int(ws.numel()), _stream(stream)))
    return ws


def sched_accept_check(rule: int, a: torch.Tensor, b: torch.Tensor, T: torch.Tensor, w3: torch.Tensor,
                       c: torch.Tensor | None = None, d: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    """The kernels' acceptance rule on given inputs (int64 a, b, c, d; float64 T; w3 as the
    int32 bits of uint32): uint8 per element, bit 0 kept, bit 1 decided by the screen."""
    k = int(a.numel())
    out = torch.empty(k, dtype=torch.uint8, device=a.device)
    _check(load_library().sched_accept_check(int(rule), k, _ptr(a), _ptr(b), _ptr(c), _ptr(d), _ptr(T), _ptr(w3),
                                             _ptr(out), _stream(stream)))
    return out
