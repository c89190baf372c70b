"""Pins of the trajectory digest and the per-chain record words of the oracle's chains.

The record's digest folds (iteration, n, t) of every accepted proposal with 64-bit FNV-1a
steps (the definition stated with sched_chains in the public header). Nothing else fixes
it, so it is pinned here from outside the oracle's C code:

- the fold itself reproduces the published FNV-1a 64-bit test vectors when it is fed the
  bytes of a string one word at a time (offset basis and prime);
- the chain loop of Algorithm 1 is walked again here, in Python, from the oracle's
  primitives (Philox block, positions, moves, replays, the two acceptance rules), and every
  record word (current key, best key and iteration, accept count, digest, start flag)
  must agree, for the fixed-size chains, the joint order / batch-size search and the
  fitted model, under both objectives and with per-level cooling;
- a wrong prime, offset, word order, or a fold of rejected proposals changes the digest.
"""
import numpy as np
import pytest

from paper_2504_14966_amd.workloads import Model, random_queue

FNV_OFFSET = 0xCBF29CE484222325
FNV_PRIME = 0x100000001B3
M64 = (1 << 64) - 1


def fnv_fold(words, d=FNV_OFFSET, prime=FNV_PRIME):
    for w in words:
        d = ((d ^ (int(w) & M64)) * prime) & M64
    return d


def as_i64(u):
    return u - (1 << 64) if u >= 1 << 63 else u


def test_fnv_published_vectors():
    # FNV-1a 64 of "", "a" and "foobar" (Fowler, Noll, Vo reference test suite)
    assert fnv_fold(b"") == 0xCBF29CE484222325
    assert fnv_fold(b"a") == 0xAF63DC4C8601EC8C
    assert fnv_fold(b"foobar") == 0x85944171F73967E8


def _better(obj, a, b):
    """Key a strictly better than b: attainment then lower latency, or G = n / t."""
    if obj == 1:
        return a[0] * b[1] > b[0] * a[1]
    return a[0] > b[0] or (a[0] == b[0] and a[1] < b[1])


def _walk(orc, n, chain, iters, T0, alpha, seed, start, obj, level_len, early_exit, propose, score):
    """Algorithm 1's loop from the oracle's primitives; returns the 8 record words."""
    st, t_ref, allmet, sn, stt = start
    state = propose("init", st)
    cn, ct = sn, stt
    bn, bt, biter, accepts, digest = cn, ct, -1, 0, FNV_OFFSET
    if early_exit and allmet:
        iters = 0
    T = T0
    for k in range(iters):
        w = [int(x) for x in orc.philox([k, chain, 0, orc.TAG_ANNEAL], [seed & 0xFFFFFFFF, seed >> 32])]
        i, j = orc.positions(n, w[1], w[2])
        cand = propose(state, (w[0], i, j))
        if cand is not None:
            nn, nt = score(cand)
            if obj == 1:
                acc = orc.accept_ratio(nn * ct - cn * nt, t_ref, ct, nt, T, w[3])
            else:
                acc = orc.accept((nn - cn) * t_ref - (nt - ct), t_ref, T, w[3])
            if acc:
                state, cn, ct = cand, nn, nt
                accepts += 1
                if _better(obj, (cn, ct), (bn, bt)):
                    bn, bt, biter = cn, ct, k
                digest = fnv_fold((k, cn, ct), digest)
        if (k + 1) % level_len == 0:
            T = T * alpha
    return [cn, ct, bn, bt, biter, accepts, as_i64(digest), int(allmet)]


def _fixed_size(orc, q, m):
    def propose(state, move):
        if isinstance(state, str):
            return np.array(move, dtype=np.uint16)
        w0, i, j = move
        return orc.swap(state, i, j) if w0 < m.swap_threshold else orc.insert(state, i, j)
    return propose, lambda perm: orc.replay(q, m, perm)


def _searched(orc, q, m, B, score_fn):
    def propose(state, move):
        if isinstance(state, str):
            return (np.array(move, dtype=np.uint16), orc.max_starts(q.n, B))
        w0, i, j = move
        perm, st = state
        op = orc.op3(w0)
        if op == 0:
            made, p, s = orc.squeeze(perm, st, B, i)
        elif op == 1:
            made, p, s = orc.delay(perm, st, B, i)
        else:
            made, p, s = q.n >= 2, orc.swap(perm, i, j), st.copy()
        return (p, s) if made else None
    return propose, lambda c: score_fn(c[0], c[1])


CASES = [(9, 3, 0, 0, 1), (12, 4, 1, 0, 1), (10, 2, 0, 1, 7), (14, 5, 1, 1, 3), (16, 16, 0, 0, 1)]


@pytest.mark.parametrize("n,B,policy,obj,L", CASES)
def test_fixed_size_chain_record(orc, n, B, policy, obj, L):
    rng = np.random.default_rng(100 + n)
    q = random_queue(rng, n, max_in=1500, max_out=40, thr_hi=700_000)
    m = Model(B, policy, p0=2000, p1=40, d0=8000, d1=300, d2=2)
    s = orc.Search(objective=obj, level_len=L)
    info = orc.start(q, m, s)
    propose, score = _fixed_size(orc, q, m)
    for chain in (0, 5):
        got = orc.anneal_chain(q, m, chain, 400, 0.7, 0.99, 2**33 + 17, start_info=info, search=s)["rec"]
        want = _walk(orc, n, chain, 400, 0.7, 0.99, 2**33 + 17, info, obj, L, 0, propose, score)
        assert got.tolist() == want, (chain, got.tolist(), want)


@pytest.mark.parametrize("n,B,obj,L", [(9, 3, 0, 1), (12, 4, 1, 5), (7, 1, 0, 1)])
def test_batch_search_chain_record(orc, n, B, obj, L):
    rng = np.random.default_rng(200 + n)
    q = random_queue(rng, n, max_in=1500, max_out=40, thr_hi=700_000)
    m = Model(B, 2, p0=2000, p1=40, d0=8000, d1=300, d2=2)
    s = orc.Search(objective=obj, level_len=L)
    info = orc.start(q, m, s)
    propose, score = _searched(orc, q, m, B, lambda p, st: orc.replay_batches(q, m, p, st))
    for chain in (1, 4):
        got = orc.anneal_chain_batches(q, m, chain, 400, 0.7, 0.99, 99, start_info=info, search=s)["rec"]
        want = _walk(orc, n, chain, 400, 0.7, 0.99, 99, info, obj, L, 0, propose, score)
        assert got.tolist() == want, (chain, got.tolist(), want)


@pytest.mark.parametrize("policy,obj,L", [(0, 0, 1), (2, 1, 10), (2, 0, 1)])
def test_fitted_model_chain_record(orc, policy, obj, L):
    rng = np.random.default_rng(300 + policy)
    n, B = 10, 4
    q = random_queue(rng, n, max_in=1500, max_out=40, thr_hi=2_000_000_000)
    fm = orc.FitModel(B, policy, **orc.TABLE2_10NS)
    s = orc.Search(objective=obj, level_len=L)
    info = orc.start_fit(q, fm, s)
    if policy == 0:
        propose, score = _fixed_size(orc, q, fm)
        score = lambda perm: orc.replay_fit(q, fm, perm)  # noqa: E731
    else:
        propose, score = _searched(orc, q, fm, B, lambda p, st: orc.replay_fit(q, fm, p, st))
    for chain in (0, 3):
        got = orc.anneal_chain_fit(q, fm, chain, 300, 50.0, 0.97, 5, search=s, start_info=info)["rec"]
        want = _walk(orc, n, chain, 300, 50.0, 0.97, 5, info, obj, L, 0, propose, score)
        assert got.tolist() == want, (chain, got.tolist(), want)


def test_early_exit_record(orc):
    rng = np.random.default_rng(5)
    q = random_queue(rng, 9, max_in=800, max_out=20)
    q.kind[:] = 2
    q.thr_us[:] = 10**9
    m = Model(3, 0, p0=2000, p1=40, d0=8000, d1=300, d2=2)
    s = orc.Search(early_exit=1)
    info = orc.start(q, m, s)
    propose, score = _fixed_size(orc, q, m)
    got = orc.anneal_chain(q, m, 0, 200, 1.0, 0.99, 0, start_info=info, search=s)["rec"]
    assert got.tolist() == _walk(orc, 9, 0, 200, 1.0, 0.99, 0, info, 0, 1, 1, propose, score)
    assert got[6] == as_i64(FNV_OFFSET)   # nothing folded


def test_digest_detects_plausible_mistakes(orc):
    """The trace of a chain folded the documented way gives its digest; folds with a wrong
    prime, offset, word order, or with rejected proposals included do not."""
    rng = np.random.default_rng(11)
    q = random_queue(rng, 12, max_in=1500, max_out=40, thr_hi=700_000)
    m = Model(4, 0, p0=2000, p1=40, d0=8000, d1=300, d2=2)
    res = orc.anneal_chain(q, m, 2, 500, 1.0, 0.99, 3, trace=True)
    tr, d = res["trace"], res["rec"][6]
    acc = [(k, int(r[1]), int(r[2])) for k, r in enumerate(tr) if r[0]]
    assert 0 < len(acc) < len(tr)
    words = [w for a in acc for w in a]
    assert as_i64(fnv_fold(words)) == d
    every = [w for k, r in enumerate(tr) for w in (k, int(r[1]), int(r[2]))]
    wrong = [fnv_fold(words, prime=0x100000001B1), fnv_fold(words, d=0),
             fnv_fold([w for a in acc for w in (a[0], a[2], a[1])]), fnv_fold(every),
             fnv_fold([w for a in acc for w in (a[1], a[2])])]
    assert all(as_i64(x) != d for x in wrong)
