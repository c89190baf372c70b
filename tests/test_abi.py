"""The C-ABI library loads, exports every symbol its header declares, and rejects bad
arguments on the host before touching a GPU."""
import ctypes as C
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER_DIR = os.path.join(ROOT, "include")


def _declared():
    names = set()
    for f in os.listdir(HEADER_DIR):
        if f.endswith(".h"):
            src = open(os.path.join(HEADER_DIR, f)).read()
            src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
            names |= set(re.findall(r"^\s*(?:const\s+)?[\w\s\*]+?\b(sched_\w+)\s*\(", src, flags=re.M))
    return names


@pytest.fixture(scope="module")
def lib():
    import paper_2504_14966_amd.sloanneal as sl
    return sl.load_library()


def test_every_declared_symbol_is_exported(lib):
    names = _declared()
    assert {"sched_eval", "sched_anneal", "sched_best", "sched_ws_bytes", "sched_strerror"} <= names
    import paper_2504_14966_amd.sloanneal as sl
    assert names == set(sl.EXPORTS)
    for nm in names:
        assert hasattr(lib, nm), nm


def test_strerror_and_ws_bytes(lib):
    assert lib.sched_strerror(0) == b"ok"
    for code in (-1, -2, -3, -4):
        assert len(lib.sched_strerror(code)) > 4
    assert lib.sched_ws_bytes(0, 1) == 0
    assert lib.sched_ws_bytes(1025, 1) == 0
    assert lib.sched_ws_bytes(8, 0) == 0
    a, b = lib.sched_ws_bytes(1024, 1), lib.sched_ws_bytes(1024, 4096)
    assert 0 < a < b and b >= 4096 * 1024 * 2 * 2 + 4096 * 64


def test_host_side_rejections_without_gpu(lib):
    import paper_2504_14966_amd.sloanneal as sl
    q = sl._Queue(0, 0, 0, 0, 0)
    m = sl._Model(4, 0, 2000, 40, 8000, 300, 2, 0, 1 << 31)
    assert lib.sched_eval(C.byref(q), C.byref(m), None, 0, None, None, None) == sl.SCHED_EINVAL
    q = sl._Queue(2000, 8, 8, 8, 8)
    assert lib.sched_eval(C.byref(q), C.byref(m), None, 0, None, None, None) == sl.SCHED_EINVAL
    q = sl._Queue(8, 8, 8, 8, 8)
    for bad in (sl._Model(0, 0, 1, 1, 1, 1, 1, 0, 0), sl._Model(65, 0, 1, 1, 1, 1, 1, 0, 0),
                sl._Model(4, 3, 1, 1, 1, 1, 1, 0, 0), sl._Model(4, 0, -1, 1, 1, 1, 1, 0, 0),
                sl._Model(4, 0, 1, 1, 1, 1, 1, 0, (1 << 32) + 1)):
        assert lib.sched_eval(C.byref(q), C.byref(bad), 8, 1, 8, None, None) == sl.SCHED_EINVAL
    assert lib.sched_eval(C.byref(q), C.byref(m), None, 1, None, None, None) == sl.SCHED_EINVAL
    assert lib.sched_eval(C.byref(q), C.byref(m), 8, -1, 8, None, None) == sl.SCHED_EINVAL
    ws = 256
    for chains, iters, T0, alpha in ((0, 1, 1.0, 0.9), (1, -1, 1.0, 0.9), (1, 1, 0.0, 0.9), (1, 1, 1.0, 0.0),
                                     (1, 1, float("nan"), 0.9), (1, 1, 1.0, float("inf"))):
        assert lib.sched_anneal(C.byref(q), C.byref(m), chains, iters, T0, alpha, 0, ws, 1 << 30, None) == \
            sl.SCHED_EINVAL
    assert lib.sched_anneal(C.byref(q), C.byref(m), 4, 1, 1.0, 0.9, 0, 257, 1 << 30, None) == sl.SCHED_EINVAL
    assert lib.sched_anneal(C.byref(q), C.byref(m), 4, 1, 1.0, 0.9, 0, ws, 100, None) == sl.SCHED_ENOSPC
    assert lib.sched_best(None, 8, 8, None) == sl.SCHED_EINVAL
    assert lib.sched_chains(None, 8, None, None, None) == sl.SCHED_EINVAL
    assert lib.sched_start_info(None, 8, 8, None) == sl.SCHED_EINVAL
    assert lib.sched_starts(None, 8, 8, 8, None) == sl.SCHED_EINVAL
    assert lib.sched_starts(256, None, None, None, None) == sl.SCHED_EINVAL
    assert lib.sched_eval_batches(C.byref(q), C.byref(m), 8, None, 1, 8, None, None) == sl.SCHED_EINVAL
    assert lib.sched_eval_batches(C.byref(q), C.byref(m), 8, 8, -1, 8, None, None) == sl.SCHED_EINVAL
    mc = sl._Model(4, 1, 2000, 40, 8000, 300, 2, 0, 1 << 31)
    assert lib.sched_eval_batches(C.byref(q), C.byref(mc), 8, 8, 1, 8, None, None) == sl.SCHED_EINVAL
    assert lib.sched_gen_perms(0, 0, 0, 1, 8, None) == sl.SCHED_EINVAL
    assert lib.sched_gen_perms(0, 8, -1, 1, 8, None) == sl.SCHED_EINVAL
    assert lib.sched_gen_perms(0, 8, 0, 0, None, None) == sl.SCHED_OK
    assert lib.sched_accept_check(2, 1, 8, 8, None, None, 8, 8, 8, None) == sl.SCHED_EINVAL
    assert lib.sched_accept_check(0, -1, 8, 8, None, None, 8, 8, 8, None) == sl.SCHED_EINVAL
    assert lib.sched_accept_check(1, 1, 8, 8, None, None, 8, 8, 8, None) == sl.SCHED_EINVAL
    assert lib.sched_accept_check(0, 0, None, None, None, None, None, None, None, None) == sl.SCHED_OK


def test_product_path_has_no_oracle_dependency():
    """The package neither imports the oracle nor names its library."""
    pkg = os.path.join(ROOT, "paper_2504_14966_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".hip", ".h", ".cpp")):
                src = open(os.path.join(dirpath, f)).read()
                assert "import oracle" not in src and "from oracle" not in src, f
                assert "liboracle" not in src and "orc_" not in src, f
