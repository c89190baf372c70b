"""The seeded synthetic queues: shapes and distributions as documented, and stable bytes."""
import json
import os

import numpy as np
import pytest

from paper_2504_14966_amd import workloads as wl

HASHES = os.path.join(os.path.dirname(__file__), "golden", "workload_hashes.json")


@pytest.mark.parametrize("idx", wl.ALL_WORKLOADS)
def test_workload_bytes_are_stable(idx):
    with open(HASHES) as f:
        want = json.load(f)["workloads"][str(idx)]
    W = wl.workload(idx)
    assert W.name == want["name"] and W.queue.n == want["n"]
    assert W.queue.sha256() == want["sha256"]


def test_lognormal_parameters():
    mu, s = wl.lognormal_params(300.0, 250.0)
    assert abs(mu - 5.4401) < 1e-4 and abs(s - 0.7262) < 1e-4
    mu, s = wl.lognormal_params(300.0, 600.0)
    assert abs(mu - 4.8991) < 1e-4 and abs(s - 1.2686) < 1e-4


def test_distributions_roughly_as_stated():
    q = wl.single_class_queue(20000, 1)
    assert 270 < q.in_len.mean() < 330 and 225 < q.out_len.mean() < 275
    assert q.in_len.min() >= 16 and q.in_len.max() <= 2048 and q.out_len.min() >= 8 and q.out_len.max() <= 1024
    q = wl.two_class_queue(20000, 1, kind_probs=(0.4, 0.3, 0.3), thr_jitter=0.25)
    frac = np.bincount(q.kind, minlength=3) / q.n
    assert abs(frac[0] - 0.4) < 0.02 and abs(frac[1] - 0.3) < 0.02
    ttft = q.thr_us[q.kind == 0]
    assert ttft.min() >= 150_000 and ttft.max() <= 375_000
    W4 = wl.workload(4)
    assert W4.queue.in_len.max() <= 8192 and W4.model.max_batch == 64 and W4.model.d1 == 250
    assert wl.workload(3).model.policy == wl.POLICY_CONTINUOUS
    assert wl.workload(5).eval_rows == 1 << 20
