// Device random numbers and the Metropolis test for gfx950.
//
// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel Random Numbers: As Easy as 1, 2, 3",
// SC'11): ten rounds of two 32x32->64 multiplies, a cross of the counter words and a key
// xor; the key advances by the two Weyl increments between rounds. Callers pass
// wave-uniform counters and keys, so the compiler keeps the whole block on the scalar unit.
//
// fast_exp_neg: e^x for x <= 0 written from the mathematics: x = k ln2 + r with
// k = floor(x / ln2 + 1/2) and |r| <= ln2 / 2, r formed with ln2 split into a 32-bit head
// (exact products with k) and a tail; e^r as its Taylor series to degree 13 evaluated by
// Horner's rule; times 2^k assembled from exponent bits. Each step is one IEEE-754
// double operation with contraction disabled, so the value is a fixed function of x.
// Below -708 (and for -inf / NaN) it returns 0.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sa {

constexpr uint32_t kTagAnneal = 0x53414E4Eu;
constexpr uint32_t kTagShuffle = 0x46495348u;

struct u32x4 {
  uint32_t x, y, z, w;
};

__device__ __forceinline__ u32x4 philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                                               uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int round = 0; round < 10; ++round) {
    const uint32_t lo0 = 0xD2511F53u * c0;
    const uint32_t hi0 = __umulhi(0xD2511F53u, c0);
    const uint32_t lo1 = 0xCD9E8D57u * c2;
    const uint32_t hi1 = __umulhi(0xCD9E8D57u, c2);
    const uint32_t n0 = hi1 ^ c1 ^ k0;
    const uint32_t n2 = hi0 ^ c3 ^ k1;
    c0 = n0;
    c1 = lo1;
    c2 = n2;
    c3 = lo0;
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  return {c0, c1, c2, c3};
}

#pragma clang fp contract(off)
__device__ __forceinline__ double fast_exp_neg(double x) {
  if (!(x >= -708.0)) return 0.0;
  if (x > 0.0) x = 0.0;
  const double kd = floor(x * 1.4426950408889634 + 0.5);
  const double r = (x - kd * 6.93147180369123816490e-01) - kd * 1.90821492927058770002e-10;
  double p = 1.0 / 6227020800.0;
  p = p * r + 1.0 / 479001600.0;
  p = p * r + 1.0 / 39916800.0;
  p = p * r + 1.0 / 3628800.0;
  p = p * r + 1.0 / 362880.0;
  p = p * r + 1.0 / 40320.0;
  p = p * r + 1.0 / 5040.0;
  p = p * r + 1.0 / 720.0;
  p = p * r + 1.0 / 120.0;
  p = p * r + 1.0 / 24.0;
  p = p * r + 1.0 / 6.0;
  p = p * r + 0.5;
  p = p * r + 1.0;
  p = p * r + 1.0;
  const int64_t k = (int64_t)kd;
  const double scale = __longlong_as_double((long long)((uint64_t)(k + 1023) << 52));
  return p * scale;
}

// Metropolis rule for a maximisation with energy n - t / t_ref, scaled by t_ref so that
// delta is an exact integer: keep any candidate that is not worse; keep a worse one
// iff u < e^(delta / (t_ref * T)), u = w3 * 2^-32.
//
// Most worse candidates are decided by a single-precision screen: with xl an estimate of
// x log2(e) (x = delta / (t_ref T)) and lu one of log2(u), g = xl - lu estimates
// log2(e^x / u). The estimates carry a relative error below 2^-20 (xl: four roundings and
// a 1-ulp reciprocal) and an absolute error below 2^-16 (lu: the 1-ulp hardware log2 of a
// value below 32 in magnitude, and the rounding of w3), and fast_exp_neg is within a few
// double ulps of e^x, so |g| > |xl| 2^-16 + 2^-10 fixes the sign of log2(E / u) with
// E = fast_exp_neg(x), i.e. the exact decision u < E. Candidates inside that band, w3 = 0,
// and denominators outside [1e-30, 1e30] take the double-precision rule itself. The
// screen needs xl > lu + 2^-10 >= -32 to accept, far above the -708 cutoff of
// fast_exp_neg, so its acceptances never fall where E = 0.
// Returns the decision in bit 0 and, in bit 1, whether the single-precision screen took it
// (0: not worse, or the double-precision rule decided).
__device__ __forceinline__ int metropolis_rule(int64_t delta, int64_t t_ref, double T, uint32_t w3) {
  if (delta >= 0) return 1;
  const double den = (double)t_ref * T;
  if (w3 != 0u && den > 1e-30 && den < 1e30) {
    const float xl = (float)delta * __builtin_amdgcn_rcpf((float)den) * 1.44269504f;
    const float lu = __builtin_amdgcn_logf((float)w3) - 32.0f;
    const float g = xl - lu;
    const float tau = fabsf(xl) * 1.52587890625e-5f + 9.765625e-4f;
    if (g > tau) return 3;
    if (g < -tau) return 2;
  }
  const double x = (double)delta / den;
  const double u = (double)w3 * (1.0 / 4294967296.0);
  return u < fast_exp_neg(x) ? 1 : 0;
}

__device__ __forceinline__ bool metropolis(int64_t delta, int64_t t_ref, double T, uint32_t w3) {
  return (metropolis_rule(delta, t_ref, T, w3) & 1) != 0;
}

// Metropolis rule for the ratio objective G = n / t, with energy G * t_ref: a candidate
// (n', t') from (n, t) changes the energy by num * t_ref / (t t'), num = n' t - n t' (exact
// int64: the device check bounds n * t below 2^63). Keep it iff num >= 0, or u < e^x with
// x = (num * t_ref) / ((t * t') * T) formed by three double operations in that order. The
// single-precision screen is the one above with the same error budget: (float) of the
// numerator and of the denominator, a 1-ulp reciprocal and two products. Bits as for
// metropolis_rule.
__device__ __forceinline__ int metropolis_ratio_rule(int64_t num, int64_t t_ref, uint64_t t, uint64_t t2, double T,
                                                     uint32_t w3) {
  if (num >= 0) return 1;
  const double a = (double)num * (double)t_ref;
  const double den = ((double)t * (double)t2) * T;
  if (w3 != 0u && den > 1e-30 && den < 1e30 && a > -1e30) {
    const float xl = (float)a * __builtin_amdgcn_rcpf((float)den) * 1.44269504f;
    const float lu = __builtin_amdgcn_logf((float)w3) - 32.0f;
    const float g = xl - lu;
    const float tau = fabsf(xl) * 1.52587890625e-5f + 9.765625e-4f;
    if (g > tau) return 3;
    if (g < -tau) return 2;
  }
  const double x = a / den;
  const double u = (double)w3 * (1.0 / 4294967296.0);
  return u < fast_exp_neg(x) ? 1 : 0;
}

__device__ __forceinline__ bool metropolis_ratio(int64_t num, int64_t t_ref, uint64_t t, uint64_t t2, double T,
                                                 uint32_t w3) {
  return (metropolis_ratio_rule(num, t_ref, t, t2, T, w3) & 1) != 0;
}

// Objective OBJ (0: attainment, then total latency; 1: ratio n / t): strict improvement.
template <int OBJ>
__device__ __forceinline__ bool obj_better(int64_t n1, uint64_t t1, int64_t n2, uint64_t t2) {
  if constexpr (OBJ == 0) {
    return n1 > n2 || (n1 == n2 && t1 < t2);
  } else {
    return n1 * (int64_t)t2 > n2 * (int64_t)t1;
  }
}

// Acceptance of a candidate that changes the key (cn, ct) by (dn, dt).
template <int OBJ>
__device__ __forceinline__ bool obj_accept(int64_t cn, uint64_t ct, int64_t dn, int64_t dt, int64_t t_ref, double T,
                                           uint32_t w3) {
  if constexpr (OBJ == 0) {
    const int64_t delta = dn * t_ref - dt;
    return metropolis(delta, t_ref, T, w3);
  } else {
    const int64_t nn = cn + dn;
    const uint64_t nt = ct + (uint64_t)dt;
    return metropolis_ratio(nn * (int64_t)ct - cn * (int64_t)nt, t_ref, ct, nt, T, w3);
  }
}

// Temperature: T0, multiplied by alpha after every `len` proposals (Algorithm 1 cools once
// per level; len = 1 is one multiply per proposal).
struct Cooling {
  double T, alpha;
  int left, len;
  __device__ __forceinline__ void step() {
    if (--left == 0) {
      left = len;
      T = T * alpha;
    }
  }
};

// Multiply-shift mapping of two 32-bit words to distinct positions i != j in [0, n).
__device__ __forceinline__ void pick_positions(int n, uint32_t w1, uint32_t w2, int &i, int &j) {
  i = (int)(((uint64_t)w1 * (uint64_t)n) >> 32);
  if (n < 2) {
    j = i;
    return;
  }
  const int jp = (int)(((uint64_t)w2 * (uint64_t)(n - 1)) >> 32);
  j = jp + (jp >= i ? 1 : 0);
}

// Proposals drawn 64 iterations at a time: lane l computes the Philox block of iteration
// k0 + l (counter (k0 + l, chain, 0, kTagAnneal)) and keeps the move packed as
// i | j << 10 | (type - 1) << 20, and, when a batch-index magic is given (at most 32
// batches), a << 21 | c << 26 with a and c the batches of min(i, j) and max(i, j); each
// iteration reads its move and acceptance word with v_readlane. Needs n <= 1024.
struct ProposalStream {
  uint32_t pk = 0, w3 = 0;
  __device__ __forceinline__ void refill(int k0, int lane, int n, uint32_t chain, uint32_t key0, uint32_t key1,
                                         uint64_t swap_thr, uint64_t bmagic) {
    const u32x4 w = philox4x32_10((uint32_t)(k0 + lane), chain, 0u, kTagAnneal, key0, key1);
    int i, j;
    pick_positions(n, w.y, w.z, i, j);
    pk = (uint32_t)i | ((uint32_t)j << 10) | (((uint64_t)w.x < swap_thr ? 0u : 1u) << 20);
    if (bmagic) {
      const uint32_t a = (uint32_t)(((uint64_t)(uint32_t)min(i, j) * bmagic) >> 32);
      const uint32_t c = (uint32_t)(((uint64_t)(uint32_t)max(i, j) * bmagic) >> 32);
      pk |= (a << 21) | (c << 26);
    }
    w3 = w.w;
  }
  // the move of iteration k (refilled when k % 64 == 0)
  __device__ __forceinline__ uint32_t packed(int k) const {
    return (uint32_t)__builtin_amdgcn_readlane((int)pk, k & 63);
  }
  __device__ __forceinline__ uint32_t word3(int k) const {
    return (uint32_t)__builtin_amdgcn_readlane((int)w3, k & 63);
  }
};

}  // namespace sa
