"""Helpers for the GPU parity tests: running the oracle over many chains in worker
processes (spawned, so they never inherit the parent's GPU state)."""
import multiprocessing as mp
import os

import numpy as np


def _search(search):
    import oracle
    return None if search is None else oracle.Search(*search)


def _chain_job(args):
    import oracle
    q, m, chain, iters, T0, alpha, seed, info, search = args
    r = oracle.anneal_chain(q, m, chain, iters, T0, alpha, seed, start_info=info, search=_search(search))
    return chain, r["rec"], r["cur"], r["best"]


def _rows_job(args):
    import oracle
    q, m, perms = args
    return oracle.eval_rows(q, m, perms)


def workers() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:
        n = os.cpu_count() or 1
    return max(1, min(n, 16))


def oracle_chains(q, m, chains, iters, T0, alpha, seed, info, search=None):
    """search: None or (objective, level_len, early_exit)."""
    jobs = [(q, m, int(c), iters, T0, alpha, seed, info, search) for c in chains]
    with mp.get_context("spawn").Pool(min(workers(), len(jobs))) as pool:
        out = pool.map(_chain_job, jobs)
    return {c: (rec, cur, best) for c, rec, cur, best in out}


def oracle_rows(q, m, perms: np.ndarray) -> np.ndarray:
    parts = np.array_split(perms, max(1, min(workers(), len(perms) // 256 + 1)))
    with mp.get_context("spawn").Pool(len(parts)) as pool:
        out = pool.map(_rows_job, [(q, m, p) for p in parts])
    return np.concatenate(out)


def _chain_batches_job(args):
    import oracle
    q, m, chain, iters, T0, alpha, seed, info, search = args
    r = oracle.anneal_chain_batches(q, m, chain, iters, T0, alpha, seed, start_info=info, search=_search(search))
    return chain, r["rec"], r["cur"], r["best"], r["cur_starts"], r["best_starts"]


def oracle_chains_batches(q, m, chains, iters, T0, alpha, seed, info, search=None):
    """Chains of the joint order / batch-size search, in worker processes."""
    jobs = [(q, m, int(c), iters, T0, alpha, seed, info, search) for c in chains]
    with mp.get_context("spawn").Pool(min(workers(), len(jobs))) as pool:
        out = pool.map(_chain_batches_job, jobs)
    return {c: dict(rec=rec, cur=cur, best=best, cur_starts=cs, best_starts=bs) for c, rec, cur, best, cs, bs in out}


def _rows_batches_job(args):
    import oracle
    q, m, perms, starts = args
    return oracle.eval_rows_batches(q, m, perms, starts)


def oracle_rows_batches(q, m, perms: np.ndarray, starts: np.ndarray) -> np.ndarray:
    k = max(1, min(workers(), len(perms) // 256 + 1))
    parts = list(zip(np.array_split(perms, k), np.array_split(starts, k)))
    with mp.get_context("spawn").Pool(len(parts)) as pool:
        out = pool.map(_rows_batches_job, [(q, m, p, s) for p, s in parts])
    return np.concatenate(out)


def _fy_rows_job(args):
    import hashlib
    import oracle
    q, m, seed, lo, hi = args
    perms = oracle.fy_perms(seed, q.n, hi - lo, row0=lo)
    return lo, hi, hashlib.sha256(np.ascontiguousarray(perms).tobytes()).hexdigest(), oracle.eval_rows(q, m, perms)


def oracle_fy_rows(q, m, seed: int, rows: int, block: int = 1 << 15):
    """Rows 0..rows-1 of the Fisher-Yates family, generated and scored by the oracle in worker
    processes: a list of (lo, hi, sha256 of the orders' bytes, (n, t) per row)."""
    jobs = [(q, m, seed, lo, min(rows, lo + block)) for lo in range(0, rows, block)]
    with mp.get_context("spawn").Pool(min(workers(), len(jobs))) as pool:
        return pool.map(_fy_rows_job, jobs)
