#!/usr/bin/env python3
"""Benchmark of the SLO-aware annealing hot path on one MI355X.

One step = one pass of the whole hot path over the burst workload (1024 requests, max
batch 64, static admission, 4096 chains x 5000 proposals, T0 2.0, alpha 0.9995):
sched_anneal (start order, every chain, cross-chain reduction) followed by sched_best.
Inputs are resident in device memory before timing starts.

Prints ONE JSON line: SA chain-iterations/s (value), plus schedule evaluations/s of the
evaluation workload (2^20 orders of 128 requests), the rates of the other annealing
workloads, the roofline of the dominant kernel and the CPU oracle baseline.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

PEAK_LANE_OPS = 256 * 4 * 16 * 2.4e9  # CUs x SIMDs x lanes x clock: int32 VALU lane-ops/s


def log(*a):
    print(*a, file=sys.stderr, flush=True)


# Algorithmic work per proposal, the method's per-unit figure: a proposal re-evaluates the
# requests from the first changed batch onward; a request whose batch changed membership
# costs about 90 int32 lane-ops (its finish offset: rank among the batch by output length
# and the segment sums, then e2e, the SLO test and its reduction share), any other
# re-evaluated request about 10 (e2e = start + offset, the SLO test, a reduction share). A
# move inside one batch changes nothing and costs nothing.
OPS_CHANGED_REQUEST = 90
OPS_REEVALUATED_REQUEST = 10
# The delta algorithm's own leaner count, reported beside it: per member of a changed batch
# two doubled pair costs (3 ops each), the newcomer's pair cost (3), the offset update (3),
# the slack and SLO test (4) and one op in each of six per-batch reductions = 22; per batch
# whose start only shifts one bounds check of 4 ops.
OPS_CHANGED_MEMBER = 22
OPS_SHIFTED_BATCH = 4
# Continuous admission (list scheduling): per admission 4 ops on each of the B list slots
# (shift, two compares, select); per event about 22 ops over the two scan passes.
OPS_CONT_PER_SLOT_ADMISSION = 4
OPS_CONT_PER_EVENT = 22


def run_studies(chains: int = 1024) -> dict:
    """The paper's parameter studies in model space (T0 / iter, output-length prediction,
    latency-predictor coefficients) at their scenarios, `chains` runs of the scheduler per
    point. Per point: label, G improvement over the arrival order (mean over chains, the
    scheduler's winner), wall ms of the point, proposals per chain."""
    from paper_2504_14966_amd import studies
    from paper_2504_14966_amd.workloads import STUDY_SCENARIOS

    def rows(pts):
        out = []
        for p in pts:
            imp = p.improvement()
            out.append([p.label, round(imp["mean"], 4), round(imp["winner"], 4), round(p.ms, 2), p.iters])
        return out

    t0 = time.perf_counter()
    res, npts = {}, 0
    for n, B in STUDY_SCENARIOS:
        for name, fn in (("T0_iter", studies.t0_iter_study), ("length", studies.length_study)):
            r = rows(fn(n, B, chains=chains))
            res[f"{name}_n{n}_b{B}"] = r
            npts += len(r)
            best = max(r, key=lambda x: x[1])
            log(f"[bench] study {name} n{n} b{B}: {len(r)} points, best mean improvement {best[1]:+.1%} ({best[0]}), "
                f"{np.mean([x[3] for x in r]):.1f} ms per point")
    r = rows(studies.coefficient_study(chains=chains))
    res["coefficients_n10_b4"] = r
    npts += len(r)
    log(f"[bench] study coefficients n10 b4: {len(r)} points, worst mean improvement "
        f"{min(x[1] for x in r):+.1%}, {np.mean([x[3] for x in r]):.1f} ms per point")
    wall = time.perf_counter() - t0
    return dict(chains_per_point=chains, points=npts, wall_s=wall, ms_per_point=wall * 1e3 / npts, results=res)


def expected_work(W) -> dict:
    """Expected work of one proposal, averaged exactly over the proposal law (i uniform, j
    uniform over the other positions, swap or insert by the swap threshold)."""
    n, B = W.queue.n, W.model.max_batch
    if W.model.policy != 0:
        b = min(B, n)
        return dict(ops=float((n - b) * OPS_CONT_PER_SLOT_ADMISSION * b + n * OPS_CONT_PER_EVENT))
    M = -(-n // B)
    sizes = np.array([min(B, n - k * B) for k in range(M)], dtype=np.float64)
    csum = np.concatenate([[0.0], np.cumsum(sizes)])
    i, j = np.meshgrid(np.arange(n), np.arange(n), indexing="ij")
    off = i != j
    a = (np.minimum(i, j) // B)[off]
    c = (np.maximum(i, j) // B)[off]
    same = a == c
    # swap: batches a and c change, batches strictly between and after shift
    sw_members = np.where(same, 0.0, sizes[a] + sizes[c])
    sw_shift = np.where(same, 0.0, (c - a - 1) + (M - 1 - c))
    # insert: batches a..c change, batches after c shift
    in_members = np.where(same, 0.0, csum[c + 1] - csum[a])
    in_shift = np.where(same, 0.0, M - 1 - c)
    # requests from the start of the first changed batch onward
    reeval = np.where(same, 0.0, n - csum[a])
    p_swap = min(W.model.swap_threshold, 1 << 32) / float(1 << 32)
    members = p_swap * sw_members.mean() + (1 - p_swap) * in_members.mean()
    shifted = p_swap * sw_shift.mean() + (1 - p_swap) * in_shift.mean()
    reevaluated = reeval.mean()
    return dict(changed_members=members, reevaluated_requests=reevaluated, shifted_batches=shifted,
                ops=OPS_CHANGED_REQUEST * members + OPS_REEVALUATED_REQUEST * (reevaluated - members),
                delta_algorithm_ops=OPS_CHANGED_MEMBER * members + OPS_SHIFTED_BATCH * shifted)


# Figures of the dominant kernel from its rocprofv3 runs, keyed by the SHA-256 of the sources
# it is compiled and launched from (every header it includes and the file that launches it);
# any other source gives null. From the counter runs over one launch of the burst workload:
#   traffic: HBM bytes per launch, FETCH_SIZE and WRITE_SIZE (KiB) scaled by the factors a
#     256 MiB device copy gives each counter in the same runs (2.0 and 1.0);
#   valu_busy: 4 x SQ_INSTS_VALU over the active cycles of all 1024 SIMDs (GRBM_GUI_ACTIVE / 8
#     per XCD), the share of cycles the vector units issue;
#   lds_bank_conflict_cycles_per_lds_instr: SQ_LDS_BANK_CONFLICT / SQ_INSTS_LDS, and
#   lds_instr_per_chain_iter: SQ_INSTS_LDS per proposal.
# From the launch itself: vgprs (the code object's count for the kernel), LDS bytes per
# workgroup (the request records, (n + 1) x 16, and 16 chains of 7,056 bytes each) and the
# waves per SIMD that are resident (4096 chains, 16 per CU in one workgroup; the LDS allows
# one such workgroup per CU, the registers five waves per SIMD).
HEADLINE_KERNEL_SOURCES = ("anneal_wave_rows.h", "anneal_wave.h", "anneal_sized.h", "anneal_static.h", "kernels.h",
                           "device_cont.h", "device_plan.h", "device_replay.h", "device_rng.h", "device_common.h",
                           "sloanneal.hip")
PROFILE_BY_SOURCE = {
    # anneal_rows_kernel<0, 16> on the burst workload: 17,420,949 B of HBM traffic (FETCH_SIZE
    # x 2.0 + WRITE_SIZE x 1.0); 441.7 VALU and 54.9 LDS instructions, 116.3 bank-conflict
    # cycles per proposal
    "1f154805f7b7b131cace531dcce6adf36ad3addcbe0c516645046ec6066bef04": {
        "traffic": 17420949, "valu_busy": 0.668, "lds_bank_conflict_cycles_per_lds_instr": 2.12,
        "lds_instr_per_chain_iter": 54.9, "vgprs": 89, "lds_bytes_per_workgroup": 129296, "waves_per_simd": 4},
}


def kernel_source_hash() -> str:
    import hashlib
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2504_14966_amd", "csrc")
    for f in HEADLINE_KERNEL_SOURCES:
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(f.encode() + b"\0" + fh.read())
    return h.hexdigest()


def measured_profile():
    """The profile figures of the headline kernel, or None when its sources changed since."""
    return PROFILE_BY_SOURCE.get(kernel_source_hash())


def time_anneal(sl, W, steps, warmup, torch):
    dq = sl.DeviceQueue.from_queue(W.queue)
    ws = sl.alloc_ws(W.queue.n, W.chains)
    stream = torch.cuda.current_stream()
    for _ in range(warmup):
        sl.sched_anneal(dq, W.model, W.chains, W.iters, W.T0, W.alpha, W.seed, ws=ws)
        sl.sched_best(ws, W.queue.n)
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    t0 = time.perf_counter()
    for s in range(steps):
        ev[s][0].record(stream)
        sl.sched_anneal(dq, W.model, W.chains, W.iters, W.T0, W.alpha, W.seed, ws=ws)
        ev[s][1].record(stream)
        perm, key = sl.sched_best(ws, W.queue.n)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    kern_ms = [a.elapsed_time(b) for a, b in ev]
    time_anneal.last_ws = ws
    return wall, kern_ms, key.cpu().tolist()


def time_eval(sl, W, reps, torch):
    dq = sl.DeviceQueue.from_queue(W.queue)
    perms = sl.sched_gen_perms(W.perm_seed, W.queue.n, W.eval_rows)
    out = torch.empty((W.eval_rows, 2), dtype=torch.int64, device="cuda")
    sl.sched_eval(dq, W.model, perms, out=out)
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    a.record(stream)
    for _ in range(reps):
        sl.sched_eval(dq, W.model, perms, out=out)
    b.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    return wall / reps, a.elapsed_time(b) / reps


def _oracle_job(args):
    import oracle
    wl, chains, iters = args
    from paper_2504_14966_amd.workloads import workload
    W = workload(wl)
    info = oracle.start(W.queue, W.model)
    t = time.perf_counter()
    recs = {}
    for c in chains:
        r = oracle.anneal_chain(W.queue, W.model, c, iters, W.T0, W.alpha, W.seed, start_info=info)
        recs[c] = (r["rec"], r["cur"], r["best"])
    return time.perf_counter() - t, recs


def cpu_model() -> str:
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


# One GPU's share of the host: at most this many worker processes, whatever the affinity
# mask shows (the host's cores are shared among the GPUs of the node).
MAX_CPU_WORKERS = 16


def cpu_baseline(wl: int, chains_per_core: int, iters: int):
    """The oracle on a bounded sample of the workload (chains_per_core whole chains per worker
    process); returns the baseline record and the oracle's per-chain results."""
    import multiprocessing as mp
    import oracle
    oracle.build(force=False)
    try:
        affinity = len(os.sched_getaffinity(0))
    except AttributeError:
        affinity = os.cpu_count() or 1
    cores = max(1, min(affinity, MAX_CPU_WORKERS))
    jobs = [(wl, list(range(k * chains_per_core, (k + 1) * chains_per_core)), iters) for k in range(cores)]
    t = time.perf_counter()
    with mp.get_context("spawn").Pool(cores) as pool:
        res = pool.map(_oracle_job, jobs)
    wall = time.perf_counter() - t
    per = [r[0] for r in res]
    recs = {c: v for r in res for c, v in r[1].items()}
    total = cores * chains_per_core * iters
    return dict(value=total / wall, unit="chain-iters/s", cores=cores, kind="oracle", affinity_cores=affinity,
                cpu_model=cpu_model(), one_core=total / sum(per),
                sample=f"workload {wl}: chains 0..{cores * chains_per_core - 1}, {iters} iterations each, "
                       f"{cores} worker processes (of {affinity} cores in the affinity mask, at most "
                       f"{MAX_CPU_WORKERS}: one GPU's share of the host), {wall:.1f} s wall "
                       f"({total / sum(per):.0f} chain-iters/s per core)"), recs


def compare_chains(sl, ws, n, chains, recs) -> dict:
    """The GPU's per-chain records and orders of the timed run against the oracle's."""
    import torch
    rec, cur, best = sl.sched_chains(ws, n, chains, perms=True)
    torch.cuda.synchronize()
    rec, cur, best = rec.cpu().numpy(), sl.as_u16(cur), sl.as_u16(best)
    bad = [c for c, (r, cu, be) in recs.items()
           if not (np.array_equal(rec[c], r) and np.array_equal(cur[c], cu) and np.array_equal(best[c], be))]
    return dict(chains_checked=len(recs), bit_exact=not bad, mismatched_chains=bad[:8])


# Oracle samples per workload (chains x iterations, or evaluation rows), as planned for the
# CPU baseline: whole chains of every annealing workload and the first 65,536 rows of the
# evaluation workload, plus the exhaustive search of the 8-request queue.
CPU_SAMPLES = {1: dict(chains=1), 2: dict(chains=64), 3: dict(chains=16), 4: dict(chains=16), 5: dict(rows=65536)}


def _oracle_sample_job(args):
    import oracle
    from paper_2504_14966_amd.workloads import workload
    wl, lo, hi = args
    W = workload(wl)
    if W.eval_rows:
        perms = oracle.fy_perms(W.perm_seed, W.queue.n, hi - lo, row0=lo)
        t = time.perf_counter()
        oracle.eval_rows(W.queue, W.model, perms)
        return time.perf_counter() - t
    info = oracle.start(W.queue, W.model)
    t = time.perf_counter()
    for c in range(lo, hi):
        oracle.anneal_chain(W.queue, W.model, c, W.iters, W.T0, W.alpha, W.seed, start_info=info)
    return time.perf_counter() - t


def cpu_all(cores: int) -> dict:
    """Oracle rates on every workload's sample: single-core and all-core (work / wall)."""
    import multiprocessing as mp
    import oracle
    from paper_2504_14966_amd.workloads import workload
    oracle.build(force=False)
    out = {}
    with mp.get_context("spawn").Pool(cores) as pool:
        for wl, smp in CPU_SAMPLES.items():
            W = workload(wl)
            units = smp.get("rows") or smp["chains"]
            per = max(1, -(-units // cores))
            jobs = [(wl, lo, min(units, lo + per)) for lo in range(0, units, per)]
            t = time.perf_counter()
            per_t = pool.map(_oracle_sample_job, jobs)
            wall = time.perf_counter() - t
            work = units if W.eval_rows else units * W.iters
            unit = "evals/s" if W.eval_rows else "chain-iters/s"
            out[W.name] = dict(unit=unit, work=work, one_core=work / sum(per_t), all_cores=work / wall,
                               processes=len(jobs), wall_s=wall)
            log(f"[bench] oracle {W.name}: {work / sum(per_t):.4g} {unit} per core, {work / wall:.4g} on {len(jobs)} processes")
        W1 = workload(1)
        t = time.perf_counter()
        oracle.brute(W1.queue, W1.model)
        out["brute_force_n8"] = dict(unit="s", orders=40320, seconds=time.perf_counter() - t)
    return out


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", type=int, default=4, choices=[1, 2, 3, 4])
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-extras", action="store_true", help="skip the other workloads")
    ap.add_argument("--no-studies", action="store_true", help="skip the parameter studies")
    ap.add_argument("--cpu-chains-per-core", type=int, default=8)
    ap.add_argument("--cpu-all", action="store_true",
                    help="also time the oracle on every workload's sample (adds about a minute)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="first run one 256 MiB device-to-device copy (reference for HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the chains are independent, so a multi-GPU run would split "
              "them and reduce one 24-byte key; run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2504_14966_amd.sloanneal as sl
    from paper_2504_14966_amd.workloads import (POLICY_STATIC, POLICY_STATIC_SEARCH, Model, multi_workload,
                                                search_workload, workload)
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    sl.load_library()

    if args.copy_calibration:
        src = torch.empty(256 << 20, dtype=torch.uint8, device="cuda").fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    W = workload(args.workload)
    log(f"[bench] workload {W.name}: {W.chains} chains x {W.iters} iters, warmup {args.warmup}, steps {args.steps}")
    wall, kern_ms, key = time_anneal(sl, W, args.steps, args.warmup, torch)
    main_ws = time_anneal.last_ws
    ms_per_step = wall * 1000.0 / args.steps
    chain_iters = W.chains * W.iters
    value = chain_iters * args.steps / wall
    k_ms = float(np.mean(kern_ms))
    work = expected_work(W)
    ops = work["ops"] * chain_iters
    achieved = ops / (k_ms * 1e-3)
    log(f"[bench] {value:.4g} chain-iters/s, anneal call {k_ms:.2f} ms, best key {key}")

    extras = {}
    if not args.no_extras:
        W5 = workload(5)
        wall5, k5 = time_eval(sl, W5, 5, torch)
        extras["eval_workload"] = dict(workload=W5.name, rows=W5.eval_rows, evals_per_s=W5.eval_rows / wall5,
                                       kernel_ms=k5)
        log(f"[bench] eval {W5.eval_rows / wall5:.4g} evals/s ({k5:.2f} ms per 2^20 rows)")
        # the same 2^20 orders with explicit batch layouts (sched_eval_batches): 1024 random
        # layouts of batch sizes uniform in 1..16, repeated over the rows
        from paper_2504_14966_amd.workloads import random_layouts
        m5 = W5.model
        ms5 = Model(m5.max_batch, POLICY_STATIC_SEARCH, m5.p0, m5.p1, m5.d0, m5.d1, m5.d2)
        lay = random_layouts(np.random.default_rng(5), 1024, W5.queue.n, m5.max_batch)
        st5 = torch.from_numpy(np.tile(lay, (W5.eval_rows // 1024, 1))).to("cuda")
        dq5 = sl.DeviceQueue.from_queue(W5.queue)
        pm5 = sl.sched_gen_perms(W5.perm_seed, W5.queue.n, W5.eval_rows)
        o5 = torch.empty((W5.eval_rows, 2), dtype=torch.int64, device="cuda")
        sl.sched_eval_batches(dq5, ms5, pm5, st5, out=o5)
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(5):
            sl.sched_eval_batches(dq5, ms5, pm5, st5, out=o5)
        b.record()
        torch.cuda.synchronize()
        msl = a.elapsed_time(b) / 5
        extras["eval_layouts"] = dict(workload="eval-n128-b16-layouts", rows=W5.eval_rows, ms=msl,
                                      evals_per_s=W5.eval_rows / (msl * 1e-3))
        log(f"[bench] eval with batch layouts {W5.eval_rows / (msl * 1e-3):.4g} evals/s ({msl:.2f} ms per 2^20 rows)")
        del st5, pm5, o5
        for wl in (1, 2, 3):
            if wl == args.workload:
                continue
            Wx = workload(wl)
            wx, kx, keyx = time_anneal(sl, Wx, 1, 1, torch)
            extras[f"anneal_{Wx.name}"] = dict(chain_iters_per_s=Wx.chains * Wx.iters / wx, ms=kx[0], best=keyx)
            log(f"[bench] {Wx.name}: {Wx.chains * Wx.iters / wx:.4g} chain-iters/s ({kx[0]:.1f} ms)")
        # the paper's own schedule and objective on the 64-request queue: T0 500, T_thres 20,
        # tau 0.95, 100 proposals per level (63 levels), G = n / t, early exit
        Wp = workload(2)
        lv = sl.sched_levels(500.0, 20.0, 0.95)
        dq = sl.DeviceQueue.from_queue(Wp.queue)
        ws = sl.alloc_ws(Wp.queue.n, Wp.chains)
        srch = sl.Search(sl.OBJ_RATIO, 100, 1)
        sl.sched_anneal(dq, Wp.model, Wp.chains, 100 * lv, 500.0, 0.95, 0, ws=ws, search=srch)
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        sl.sched_anneal(dq, Wp.model, Wp.chains, 100 * lv, 500.0, 0.95, 0, ws=ws, search=srch)
        b.record()
        _, keyp = sl.sched_best(ws, Wp.queue.n)
        torch.cuda.synchronize()
        msp = a.elapsed_time(b)
        extras["anneal_paper_schedule_mix-n64-b16"] = dict(chains=Wp.chains, iters=100 * lv, ms=msp,
                                                          chain_iters_per_s=Wp.chains * 100 * lv / (msp * 1e-3),
                                                          best=keyp.cpu().tolist())
        log(f"[bench] paper schedule (G, 63 levels x 100) on mix-n64: {Wp.chains * 100 * lv / (msp * 1e-3):.4g} "
            f"chain-iters/s ({msp:.1f} ms), best {keyp.cpu().tolist()}")
        # several serving instances: the 1024-request queue assigned to 8 instances, every
        # instance's chains in one launch, against the instances annealed one after another
        Wm = multi_workload()
        Im = Wm.extra["instances"]
        dqm = sl.DeviceQueue.from_queue(Wm.queue)
        capm = torch.tensor(Wm.extra["capacity"], dtype=torch.int64, device="cuda")
        inst = sl.sched_assign(dqm, capm)
        mws = sl.sched_anneal_multi(dqm, Wm.model, inst, Im, Wm.chains, Wm.iters, Wm.T0, Wm.alpha, Wm.seed)
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        inst = sl.sched_assign(dqm, capm)
        sl.sched_anneal_multi(dqm, Wm.model, inst, Im, Wm.chains, Wm.iters, Wm.T0, Wm.alpha, Wm.seed, mws=mws)
        sl.sched_multi_best(mws)
        b.record()
        torch.cuda.synchronize()
        ms_one = a.elapsed_time(b)
        inst_h = inst.cpu().numpy()
        subs = []
        for k in range(Im):
            ids = np.flatnonzero(inst_h == k)
            from paper_2504_14966_amd.workloads import Queue
            subs.append(sl.DeviceQueue.from_queue(Queue(Wm.queue.in_len[ids], Wm.queue.out_len[ids], Wm.queue.kind[ids],
                                                        Wm.queue.thr_us[ids])))
        wss = [sl.alloc_ws(sq.n, Wm.chains) for sq in subs]
        for sq, w in zip(subs, wss):
            sl.sched_anneal(sq, Wm.model, Wm.chains, Wm.iters, Wm.T0, Wm.alpha, Wm.seed, ws=w)
        torch.cuda.synchronize()
        a.record()
        for sq, w in zip(subs, wss):
            sl.sched_anneal(sq, Wm.model, Wm.chains, Wm.iters, Wm.T0, Wm.alpha, Wm.seed, ws=w)
        b.record()
        torch.cuda.synchronize()
        ms_seq = a.elapsed_time(b)
        ci = Im * Wm.chains * Wm.iters
        extras[f"anneal_{Wm.name}"] = dict(instances=Im, chains_per_instance=Wm.chains, iters=Wm.iters,
                                           requests_per_instance=np.bincount(inst_h, minlength=Im).tolist(),
                                           one_launch_ms=ms_one, chain_iters_per_s=ci / (ms_one * 1e-3),
                                           one_after_another_ms=ms_seq)
        log(f"[bench] {Wm.name}: {ci / (ms_one * 1e-3):.4g} chain-iters/s in one launch ({ms_one:.1f} ms, "
            f"assignment included); instances one after another {ms_seq:.1f} ms")
        # the paper's multi-instance setting in model space: the same 10 requests replicated on
        # each of I instances (max batch 4), the paper's schedule (G, T0 500 cooled by 0.95 to
        # 20, 100 proposals per level, early exit), 1024 chains per instance; all instances in
        # one launch against one sched_anneal per instance
        from paper_2504_14966_amd.workloads import Queue, two_class_queue
        q10 = two_class_queue(10, 0)
        m10 = Model(4, POLICY_STATIC, 2000, 40, 8000, 300, 2)
        lv10 = sl.sched_levels(500.0, 20.0, 0.95)
        s10 = sl.Search(sl.OBJ_RATIO, 100, 1)
        rep = {}
        for I in (1, 2, 4, 8):
            qI = Queue(np.tile(q10.in_len, I), np.tile(q10.out_len, I), np.tile(q10.kind, I), np.tile(q10.thr_us, I))
            dqI = sl.DeviceQueue.from_queue(qI)
            instI = torch.tensor(np.repeat(np.arange(I, dtype=np.int32), 10), device="cuda")
            mwsI = sl.sched_anneal_multi(dqI, m10, instI, I, 1024, 100 * lv10, 500.0, 0.95, 0, search=s10)
            torch.cuda.synchronize()
            a.record()
            sl.sched_anneal_multi(dqI, m10, instI, I, 1024, 100 * lv10, 500.0, 0.95, 0, search=s10, mws=mwsI)
            sl.sched_multi_best(mwsI)
            b.record()
            torch.cuda.synchronize()
            ms1 = a.elapsed_time(b)
            d10 = sl.DeviceQueue.from_queue(q10)
            w10 = sl.alloc_ws(10, 1024)
            sl.sched_anneal(d10, m10, 1024, 100 * lv10, 500.0, 0.95, 0, ws=w10, search=s10)
            torch.cuda.synchronize()
            a.record()
            for _ in range(I):
                sl.sched_anneal(d10, m10, 1024, 100 * lv10, 500.0, 0.95, 0, ws=w10, search=s10)
                sl.sched_best(w10, 10)
            b.record()
            torch.cuda.synchronize()
            rep[I] = dict(one_launch_ms=ms1, one_after_another_ms=a.elapsed_time(b))
        extras["multi_replicated_n10_b4_paper_schedule"] = dict(chains_per_instance=1024, iters=100 * lv10,
                                                                 by_instances=rep)
        log("[bench] 10 requests replicated on 1/2/4/8 instances, paper schedule: one launch " +
            "/".join(f"{rep[I]['one_launch_ms']:.2f}" for I in rep) + " ms; one after another " +
            "/".join(f"{rep[I]['one_after_another_ms']:.2f}" for I in rep) + " ms")
        # the fitted model taken literally (Table 2 in units of 10 ns) on 256 chat / code
        # requests with the paper's SLOs (code: e2e 30 s; chat: TTFT 10 s and TPOT 50 ms),
        # batch sizes searched (max 16), 2048 chains x 2000 proposals
        from paper_2504_14966_amd.workloads import TABLE2_10NS, chat_code_queue_10ns
        qf, thr2 = chat_code_queue_10ns(256, 0)
        fit = sl.FitModel(16, sl.POLICY_STATIC_SEARCH, **TABLE2_10NS)
        dqf, t2 = sl.DeviceQueue.from_queue(qf), sl.thr_to_device(thr2)
        wsf = sl.alloc_ws(qf.n, 2048)
        sl.sched_anneal_fit(dqf, fit, 2048, 2000, 1.0, 0.999, 0, tpot_thr=t2, ws=wsf)
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        sl.sched_anneal_fit(dqf, fit, 2048, 2000, 1.0, 0.999, 0, tpot_thr=t2, ws=wsf)
        b.record()
        _, keyf = sl.sched_best(wsf, qf.n)
        torch.cuda.synchronize()
        msf = a.elapsed_time(b)
        extras["anneal_fit-table2-chatcode-n256-b16-search"] = dict(ms=msf, chain_iters_per_s=2048 * 2000 / (msf * 1e-3),
                                                                    best=keyf.cpu().tolist(), time_unit="10 ns")
        log(f"[bench] fitted model, chat/code n256 batch sizes searched: {2048 * 2000 / (msf * 1e-3):.4g} "
            f"chain-iters/s ({msf:.1f} ms), best {keyf.cpu().tolist()}")
        # the joint order / batch-size search (squeeze, delay and swap moves) on the same queues
        for wl in (2, 4):
            Wx = search_workload(wl)
            wx, kx, keyx = time_anneal(sl, Wx, 2, 1, torch)
            extras[f"anneal_{Wx.name}"] = dict(chain_iters_per_s=2 * Wx.chains * Wx.iters / wx, ms=float(np.mean(kx)),
                                               best=keyx)
            log(f"[bench] {Wx.name}: {2 * Wx.chains * Wx.iters / wx:.4g} chain-iters/s ({np.mean(kx):.1f} ms), "
                f"best {keyx}")
        if not args.no_studies:
            extras["studies"] = run_studies()

    cpu = None
    if args.cpu_all:
        try:
            ncores = max(1, min(len(os.sched_getaffinity(0)), MAX_CPU_WORKERS))
        except AttributeError:
            ncores = max(1, min(os.cpu_count() or 1, MAX_CPU_WORKERS))
        extras["oracle_all_workloads"] = cpu_all(ncores)
    if not args.no_cpu:
        log("[bench] CPU oracle baseline ...")
        cpu, recs = cpu_baseline(args.workload, args.cpu_chains_per_core, W.iters)
        log(f"[bench] oracle {cpu['value']:.4g} chain-iters/s on {cpu['cores']} cores ({cpu['cpu_model']})")
        cpu["parity"] = compare_chains(sl, main_ws, W.queue.n, W.chains, recs)
        log(f"[bench] oracle chains against the timed run's GPU records: {cpu['parity']}")

    prof = measured_profile()
    line = {
        "metric": "SA chain-iterations/s",
        "value": value,
        "unit": "chain-iters/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int64",
        "data": "synthetic",
        "config": {"workload": W.name, "requests": W.queue.n, "max_batch": W.model.max_batch,
                   "policy": "static" if W.model.policy == 0 else "continuous", "chains": W.chains,
                   "iters": W.iters, "T0": W.T0, "alpha": W.alpha, "parallelism": "chains"},
        "roofline": {"bound": "alu", "achieved": achieved / 1e12, "peak": PEAK_LANE_OPS / 1e12, "unit": "TOP/s",
                     "frac": achieved / PEAK_LANE_OPS, "traffic": (prof or {}).get("traffic"),
                     "rocprof": prof,
                     "delta_algorithm_frac": (work.get("delta_algorithm_ops", 0.0) * chain_iters / (k_ms * 1e-3))
                                             / PEAK_LANE_OPS,
                     "kernel": "anneal_rows_kernel", "kernel_ms": k_ms,
                     "algo_lane_ops_per_chain_iter": work["ops"], "work_per_chain_iter": work},
        "cpu_baseline": cpu,
        "extras": extras,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
