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
