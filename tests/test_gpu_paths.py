"""GPU parity of every kernel path the host dispatch can choose, against the oracle.

The library picks a kernel from the queue and model: the static delta kernels (32-bit
finish offsets; batch records in LDS for B <= 32, in lane-per-batch registers for B > 32,
with every member's SLO limit in registers too when the whole timeline fits 32 bits),
the continuous list-scheduling replay (total output below 2^22 tokens), the continuous
event loop (32-bit event arithmetic), or the general full-replay kernels (64-bit
everything). Each case below is built so that its
sizes and coefficients fall on one path; all must agree with the oracle bit for bit.
"""
import os
import sys
import zlib

import numpy as np
import pytest

sys.path.insert(0, os.path.dirname(__file__))
from gpu_helpers import oracle_chains  # noqa: E402

from paper_2504_14966_amd.workloads import Model, Queue  # noqa: E402

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sl():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2504_14966_amd.sloanneal as m
    m.load_library()
    return m


def _queue(rng, n, in_lo, in_hi, out_lo, out_hi, thr_hi):
    return Queue(rng.integers(in_lo, in_hi + 1, n).astype(np.uint16), rng.integers(out_lo, out_hi + 1, n).astype(np.uint16),
                 rng.integers(0, 3, n).astype(np.uint8), rng.integers(0, thr_hi, n).astype(np.uint32))


CASES = {
    # static, B = 1 over 1024 requests: delta kernel with one lane per batch
    "static_b1_n1024": (lambda r: _queue(r, 1024, 16, 2048, 1, 6, 4_000_000_000), Model(1, 0, 2000, 40, 8000, 300, 2), 8, 150),
    # static, one batch per wave (B > 32) with a ragged last batch: lane-per-batch kernel
    "static_wave_ragged": (lambda r: _queue(r, 150, 16, 2048, 1, 300, 4_000_000_000), Model(40, 0, 2000, 40, 8000, 300, 2), 8, 400),
    # static, one batch per wave with a timeline beyond 2^32 (every finish offset still
    # within 32 bits): the lane-per-batch kernel without the registers of member limits
    "static_wave_wide_time": (lambda r: _queue(r, 300, 16, 2048, 1000, 3000, 4_000_000_000), Model(40, 0, 2000, 40, 8000, 300, 2), 4, 120),
    # static, B > 32 and B > n: a single batch, every move keeps the objective
    "static_wave_one_batch": (lambda r: _queue(r, 50, 16, 2048, 1, 300, 4_000_000_000), Model(64, 0, 2000, 40, 8000, 300, 2), 4, 100),
    # static, d2 so large that pair costs exceed 24 bits: general full-replay kernel
    "static_wide": (lambda r: _queue(r, 48, 16, 2048, 8, 300, 4_000_000_000), Model(8, 0, 2000, 40, 8000, 300, 1 << 22), 16, 300),
    # continuous, total output above 2^22 tokens: event loop instead of list scheduling
    "cont_event_loop": (lambda r: _queue(r, 128, 16, 2048, 40000, 65535, 4_000_000_000), Model(64, 1, 2000, 40, 8000, 300, 2), 4, 40),
    # continuous, context cost above 32 bits: general 64-bit event loop
    "cont_wide": (lambda r: _queue(r, 24, 16, 2048, 4, 40, 4_000_000_000), Model(6, 1, 2000, 40, 8000, 300, 1 << 25), 16, 300),
    # continuous, list scheduling with ties (equal output lengths) and B > n
    "cont_ls_ties": (lambda r: _queue(r, 40, 16, 64, 5, 7, 3_000_000), Model(16, 1, 2000, 40, 8000, 300, 2), 16, 400),
    "cont_ls_b_gt_n": (lambda r: _queue(r, 20, 16, 2048, 8, 200, 3_000_000), Model(32, 1, 2000, 40, 8000, 300, 2), 8, 300),
    # continuous, list scheduling with more than 32 running requests (one-lane pop register
    # instead of the sliding window), including a full 64-lane list
    "cont_ls_b48": (lambda r: _queue(r, 100, 16, 2048, 4, 200, 3_000_000), Model(48, 1, 2000, 40, 8000, 300, 2), 8, 300),
    "cont_ls_b64": (lambda r: _queue(r, 150, 16, 2048, 4, 200, 3_000_000), Model(64, 1, 2000, 40, 8000, 300, 2), 8, 200),
    # continuous, list scheduling with a timeline longer than 2^32 us (64-bit segment sums)
    "cont_ls_wide_time": (lambda r: _queue(r, 40, 16, 2048, 20000, 60000, 4_000_000_000), Model(8, 1, 2000, 40, 8000, 300, 2), 4, 60),
    # continuous, two proposals per round: one running request (63 admissions per window
    # chunk, a ragged second chunk), a single admission after the initial group, a single
    # request (every move is the identity); odd proposal counts end on a lone proposal
    "cont_spec_b1": (lambda r: _queue(r, 70, 16, 2048, 1, 200, 3_000_000), Model(1, 1, 2000, 40, 8000, 300, 2), 4, 301),
    "cont_spec_b32_n33": (lambda r: _queue(r, 33, 16, 2048, 1, 200, 3_000_000), Model(32, 1, 2000, 40, 8000, 300, 2), 4, 257),
    "cont_spec_one": (lambda r: _queue(r, 1, 16, 2048, 1, 200, 3_000_000), Model(4, 1, 2000, 40, 8000, 300, 2), 2, 65),
    # 48 running with a timeline beyond 2^32: the two-proposal kernel is listed (first) and
    # refused on the device, the single-proposal list-scheduling kernel runs
    "cont_ls_b48_wide_time": (lambda r: _queue(r, 60, 16, 2048, 20000, 60000, 4_000_000_000),
                              Model(48, 1, 2000, 40, 8000, 300, 2), 4, 60),
    # more chains than the GPU holds at once: later workgroups start as earlier ones end
    "cont_spec_many_chains": (lambda r: _queue(r, 40, 16, 2048, 1, 200, 3_000_000), Model(8, 1, 2000, 40, 8000, 300, 2),
                              2500, 60),
}


# the candidate that must run, for cases where the order of candidates is the point: under
# static admission with B > 32, the kernel with the member limits in registers comes first
# and needs a 32-bit timeline; the plain lane-per-batch kernel follows it. Under continuous
# admission the kernel scoring two proposals per round comes first and needs 32-bit times;
# the single-proposal list-scheduling kernel follows it
SELECTED = {"static_wave_ragged": 0, "static_wave_wide_time": 1, "cont_ls_ties": 0, "cont_ls_b_gt_n": 0,
            "cont_spec_b1": 0, "cont_spec_b32_n33": 0, "cont_spec_one": 0, "cont_spec_many_chains": 0,
            "cont_ls_wide_time": 1, "cont_ls_b48": 0, "cont_ls_b64": 0, "cont_ls_b48_wide_time": 1}


@pytest.mark.parametrize("name", sorted(CASES))
def test_eval_path(sl, orc, name):
    mk, m, _, _ = CASES[name]
    rng = np.random.default_rng(zlib.crc32(name.encode()))
    q = mk(rng)
    rows = 6
    perms = np.stack([rng.permutation(q.n) for _ in range(rows)]).astype(np.uint16)
    dq = sl.DeviceQueue.from_queue(q)
    out, det = sl.sched_eval(dq, m, sl.perms_to_device(perms), detail=True)
    out, det = out.cpu().numpy(), det.cpu().numpy()
    for r in range(rows):
        nn, tt, ttft, e2e = orc.replay(q, m, perms[r], detail=True)
        assert out[r].tolist() == [nn, tt], (name, r)
        assert np.array_equal(det[r, :, 0], ttft) and np.array_equal(det[r, :, 1], e2e), (name, r)


@pytest.mark.parametrize("name", sorted(CASES))
def test_anneal_path(sl, orc, name):
    import torch
    mk, m, chains, iters = CASES[name]
    rng = np.random.default_rng(zlib.crc32(name.encode()))
    q = mk(rng)
    dq = sl.DeviceQueue.from_queue(q)
    ws = sl.sched_anneal(dq, m, chains, iters, 0.7, 0.99, 11)
    rec, cur, best = sl.sched_chains(ws, q.n, chains, perms=True)
    status = sl.sched_status(ws).cpu().tolist()
    torch.cuda.synchronize()
    assert status[0] == 0, (name, status)
    if name in SELECTED:
        assert status[2] == SELECTED[name], (name, status)
    rec, cur, best = rec.cpu().numpy(), sl.as_u16(cur), sl.as_u16(best)
    info = orc.start(q, m)
    want = oracle_chains(q, m, list(range(chains)), iters, 0.7, 0.99, 11, info)
    for c in range(chains):
        wrec, wcur, wbest = want[c]
        assert rec[c].tolist() == wrec.tolist(), (name, c)
        assert cur[c].tolist() == wcur.tolist() and best[c].tolist() == wbest.tolist(), (name, c)
