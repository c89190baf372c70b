"""Integer identities the GPU kernels rely on, checked exhaustively on the CPU."""
import numpy as np


def test_batch_index_magic_division():
    """Batch index p / B as (p * (floor(2^32 / B) + 1)) >> 32 for every B <= 64 and p < 2^16
    (for B = 1 the multiplier is 2^32 + 1, which needs 64 bits)."""
    p = np.arange(1 << 16, dtype=np.uint64)
    for B in range(1, 65):
        m = np.uint64((1 << 32) // B + 1)
        assert np.array_equal((p * m) >> np.uint64(32), p // np.uint64(B)), B


def test_doubled_pair_cost_identity():
    """2 * (d1*mu + d2*(l*mu + mu(mu+1)/2)) == mu * (e + d2*mu) with e = 2(d1 + d2 l) + d2."""
    rng = np.random.default_rng(0)
    for _ in range(20000):
        d1, d2, l, mu = (int(x) for x in rng.integers(0, [500, 8, 65536, 65536]))
        e = 2 * (d1 + d2 * l) + d2
        assert 2 * (d1 * mu + d2 * (l * mu + mu * (mu + 1) // 2)) == mu * (e + d2 * mu)


def test_segment_cost_closed_form():
    """Sum over u = 1..s of (d0 + d1 b + d2 (C + b u)) == s (d0 + d1 b + d2 C) + d2 b s (s + 1) / 2."""
    rng = np.random.default_rng(1)
    for _ in range(2000):
        d0, d1, d2, b, C, s = (int(x) for x in rng.integers(0, [9000, 400, 4, 65, 1 << 20, 3000]))
        assert sum(d0 + d1 * b + d2 * (C + b * u) for u in range(1, s + 1)) == \
            s * (d0 + d1 * b + d2 * C) + d2 * b * s * (s + 1) // 2


def test_metropolis_single_precision_screen(orc):
    """The kernels decide most worse candidates with a single-precision estimate g of
    log2(e^x / u) and fall back to the double-precision rule when |g| <= |xl| 2^-16 + 2^-10.
    Emulated here in float32 with the estimates pushed to the edges of their stated error
    (xl relative 2^-20, lu absolute 2^-16), every decision the screen takes must equal the
    oracle's exact rule (u < det_exp(delta / (t_ref T)))."""
    rng = np.random.default_rng(7)
    n = 20000
    t_ref = rng.integers(1, 1 << 40, n)
    T = np.exp(rng.uniform(np.log(1e-6), np.log(10.0), n))
    x_target = -np.exp(rng.uniform(np.log(1e-6), np.log(60.0), n))
    delta = np.minimum(np.floor(x_target * t_ref * T), -1).astype(np.int64)
    w3 = rng.integers(1, 1 << 32, n, dtype=np.uint64)
    # half the samples sit next to the boundary u = e^x
    near = rng.random(n) < 0.5
    x = delta / (t_ref.astype(np.float64) * T)
    w_edge = np.clip(np.floor(np.exp(x) * 2.0**32) + rng.integers(-3, 4, n), 1, (1 << 32) - 1)
    w3 = np.where(near, w_edge.astype(np.uint64), w3)
    den = (t_ref.astype(np.float64) * T)
    xl = (delta.astype(np.float32) * (np.float32(1.0) / den.astype(np.float32))) * np.float32(1.44269504)
    lu = np.log2(w3.astype(np.float32)) - np.float32(32.0)
    tau = np.abs(xl) * np.float32(1.52587890625e-5) + np.float32(9.765625e-4)
    decided = np.zeros(n, np.int64)
    for s in range(n):
        want = orc.accept(int(delta[s]), int(t_ref[s]), float(T[s]), int(w3[s]))
        for ex in (1 - 2.0**-20, 1 + 2.0**-20):
            for el in (-2.0**-16, 2.0**-16):
                g = np.float32(xl[s] * ex) - np.float32(lu[s] + el)
                if g > tau[s]:
                    assert want, (s, int(delta[s]), int(t_ref[s]), T[s], int(w3[s]))
                    decided[s] += 1
                elif g < -tau[s]:
                    assert not want, (s, int(delta[s]), int(t_ref[s]), T[s], int(w3[s]))
                    decided[s] += 1
    # away from the boundary the screen decides nearly everything
    assert decided[~near].sum() > 0.99 * 4 * (~near).sum()


def test_pair_costs_are_even():
    """mu (e + d2 mu) with e = 2 (d1 + d2 l) + d2 is even: 2 mu (d1 + d2 l) + d2 mu (mu + 1).
    The one-batch-per-wave kernels halve a newcomer's pair-cost sum and its correction
    w(e, e) - w(o, e) one by one, which is exact only for even terms."""
    rng = np.random.default_rng(11)
    d1 = rng.integers(0, 1 << 12, 200000, dtype=np.int64)
    d2 = rng.integers(0, 1 << 6, 200000, dtype=np.int64)
    l = rng.integers(0, 1 << 16, 200000, dtype=np.int64)
    mu = rng.integers(0, 1 << 16, 200000, dtype=np.int64)
    e = 2 * (d1 + d2 * l) + d2
    assert np.all((mu * (e + d2 * mu)) % 2 == 0)
    for dd1 in range(4):  # exhaustive on a small grid, odd and even parameters alike
        for dd2 in range(4):
            for ll in range(8):
                ee = 2 * (dd1 + dd2 * ll) + dd2
                assert all((m * (ee + dd2 * m)) % 2 == 0 for m in range(64))


def _limit_of_u32(kind, thr, lout, P, F):
    """A member's limit as the one-batch-per-wave kernel with registers of limits forms it:
    the staged record holds thr1 = min(thr', 2^32 - 2) + 1 (thr' = thr, or thr * l_out
    saturated at 2^32 - 1 for TPOT); met iff the batch start is below the limit."""
    u = np.uint64
    thr_st = np.where(kind == 1, np.minimum(thr.astype(u) * lout.astype(u), u(0xFFFFFFFF)), thr.astype(u))
    thr1 = (np.minimum(thr_st, u(0xFFFFFFFE)) + u(1)).astype(np.uint32)
    off = np.where(kind == 0, P, F).astype(np.int64)
    by_start = np.maximum(thr1.astype(np.int64) - off, 0).astype(np.uint32)  # saturating subtract
    tpot = np.where((F.astype(np.int64) - P.astype(np.int64)) < thr1.astype(np.int64), 0xFFFFFFFF, 0).astype(np.uint32)
    return np.where(kind == 1, tpot, by_start)


def test_limit_rows_decide_like_the_slo_test():
    """S < limit equals the SLO test of the Problem Formulation (TTFT = S + P <= thr,
    e2e = S + F <= thr, TPOT = (e2e - TTFT) / l_out <= thr) whenever the kernel's width
    conditions hold: every time on the timeline below 2^32 - 2 (S + F), thresholds up to
    2^32 - 2, finish offsets below 2^32 - 1. Random cases and the edges: starts at and
    around each threshold, the largest thresholds, TPOT products that saturate."""
    rng = np.random.default_rng(12)
    n = 400000
    top = (1 << 32) - 3  # largest time on the timeline
    kind = rng.integers(0, 3, n)
    lout = rng.integers(1, 1 << 16, n)
    F = rng.integers(0, 1 << 32, n) % (top + 1)
    P = rng.integers(0, 1 << 32, n) % (F + 1)  # the batch prefill is part of every offset
    S = rng.integers(0, 1 << 32, n) % (top - F + 1)
    thr = rng.integers(0, 0xFFFFFFFE + 1, n)
    # edges: thresholds at the start plus the offset, one below and one above, and the largest
    edge = rng.integers(0, 5, n)
    off = np.where(kind == 0, P, F)
    tp = (F - P + lout - 1) // lout  # the smallest TPOT threshold that is met
    near = np.where(kind == 1, tp, S + off)
    thr = np.where(edge == 1, near, thr)
    thr = np.where(edge == 2, np.maximum(near - 1, 0), thr)
    thr = np.where(edge == 3, np.minimum(near + 1, 0xFFFFFFFE), thr)
    thr = np.where(edge == 4, 0xFFFFFFFE, thr)
    thr = np.minimum(thr, 0xFFFFFFFE)
    lim = _limit_of_u32(kind, thr, lout, P, F)
    got = S < lim.astype(np.int64)
    ttft, e2e = S + P, S + F
    want = np.where(kind == 0, ttft <= thr, np.where(kind == 2, e2e <= thr, (e2e - ttft) <= thr * lout))
    assert np.array_equal(got, want)
    assert want.any() and (~want).any()
