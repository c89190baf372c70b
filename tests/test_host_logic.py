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
