/* Oracle random numbers and the Metropolis test -- TEST INFRASTRUCTURE ONLY (see oracle.h).
 *
 * Philox4x32-10: the counter-based generator of Salmon, Moraes, Dror and Shaw,
 * "Parallel Random Numbers: As Easy as 1, 2, 3" (SC'11). Ten rounds; each round
 * multiplies counter words 0 and 2 by the two round multipliers, and the key is
 * bumped by the two Weyl constants between rounds.
 *
 * det_exp: exp(x) written from the mathematics. x = k*ln2 + r with k = round(x/ln2)
 * and |r| <= ln2/2 (Cody and Waite's two-constant reduction, ln2 split into a short
 * high part and a low correction); exp(r) is the Taylor series to degree 13 in
 * Horner form, and the result is scaled by 2^k built from its exponent bits. Every
 * operation is a single IEEE-754 double operation (this file is compiled with
 * -ffp-contract=off), so the result is a fixed function of x.
 *
 * The Metropolis rule: the paper's acceptance test (Algorithm 1) is written so that a
 * worse candidate is accepted when exp(-(f_new - f)/T) < rand, which never holds for a
 * worse candidate; this oracle takes the standard rule for a maximisation, accept
 * with probability exp((f_new - f)/T), which is the behaviour the section "Priority
 * Mapping Algorithm" describes (higher temperature, likelier acceptance of a worse
 * solution). With f = n - t / t_ref, (f_new - f) * t_ref = delta is an exact int64.
 */
#include "oracle.h"
#include <string.h>

#define PHILOX_M0 0xD2511F53u
#define PHILOX_M1 0xCD9E8D57u
#define PHILOX_W0 0x9E3779B9u
#define PHILOX_W1 0xBB67AE85u

void orc_philox(const uint32_t ctr_in[4], const uint32_t key_in[2], uint32_t out[4]) {
  uint32_t c[4], k[2];
  memcpy(c, ctr_in, sizeof c);
  memcpy(k, key_in, sizeof k);
  for (int round = 0; round < 10; round++) {
    if (round > 0) {
      k[0] += PHILOX_W0;
      k[1] += PHILOX_W1;
    }
    uint64_t p0 = (uint64_t)PHILOX_M0 * c[0];
    uint64_t p1 = (uint64_t)PHILOX_M1 * c[2];
    uint32_t n0 = (uint32_t)(p1 >> 32) ^ c[1] ^ k[0];
    uint32_t n1 = (uint32_t)p1;
    uint32_t n2 = (uint32_t)(p0 >> 32) ^ c[3] ^ k[1];
    uint32_t n3 = (uint32_t)p0;
    c[0] = n0; c[1] = n1; c[2] = n2; c[3] = n3;
  }
  memcpy(out, c, sizeof c);
}

double orc_det_exp(double x) {
  const double inv_ln2 = 1.4426950408889634;        /* 1/ln 2 */
  const double ln2_hi = 6.93147180369123816490e-01; /* ln 2 rounded to 32 significant bits */
  const double ln2_lo = 1.90821492927058770002e-10; /* ln 2 - ln2_hi */
  if (!(x >= -708.0)) return 0.0;                   /* also -inf and NaN */
  if (x > 0.0) x = 0.0;
  double kd = __builtin_floor(x * inv_ln2 + 0.5);
  double r = (x - kd * ln2_hi) - kd * ln2_lo;
  /* Taylor coefficients 1/j!, j = 13 .. 0 */
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
  int64_t k = (int64_t)kd;
  uint64_t bits = (uint64_t)(k + 1023) << 52;
  double scale;
  memcpy(&scale, &bits, sizeof scale);
  return p * scale;
}

int orc_accept(int64_t delta, int64_t t_ref, double T, uint32_t w3) {
  if (delta >= 0) return 1;
  double x = (double)delta / ((double)t_ref * T);
  double u = (double)w3 * (1.0 / 4294967296.0);
  return u < orc_det_exp(x);
}

int orc_accept_ratio(int64_t num, int64_t t_ref, int64_t t, int64_t t2, double T, uint32_t w3) {
  if (num >= 0) return 1;
  double a = (double)num * (double)t_ref;
  double den = ((double)t * (double)t2) * T;
  double x = a / den;
  double u = (double)w3 * (1.0 / 4294967296.0);
  return u < orc_det_exp(x);
}

/* The two acceptance rules over arrays (rule 0: orc_accept(a, b, T, w3); rule 1:
 * orc_accept_ratio(a, b, c, d, T, w3)), one decision per element. */
void orc_accept_many(int32_t rule, int64_t k, const int64_t *a, const int64_t *b, const int64_t *c,
                     const int64_t *d, const double *T, const uint32_t *w3, uint8_t *out) {
  for (int64_t r = 0; r < k; r++) {
    out[r] = (uint8_t)(rule == 1 ? orc_accept_ratio(a[r], b[r], c[r], d[r], T[r], w3[r])
                                 : orc_accept(a[r], b[r], T[r], w3[r]));
  }
}

int32_t orc_levels(double T0, double T_thres, double tau) {
  int32_t levels = 0;
  double T = T0;
  do {
    levels++;
    T = T * tau;
  } while (T >= T_thres && levels < (1 << 30));
  return levels;
}

void orc_fy_perm(uint64_t seed, int32_t n, uint32_t idx, uint16_t *perm) {
  uint32_t key[2] = { (uint32_t)seed, (uint32_t)(seed >> 32) };
  for (int32_t p = 0; p < n; p++) perm[p] = (uint16_t)p;
  for (int32_t k = n - 1; k >= 1; k--) {
    uint32_t ctr[4] = { (uint32_t)k >> 2, idx, 1u, (uint32_t)ORC_TAG_FY };
    uint32_t w[4];
    orc_philox(ctr, key, w);
    uint32_t j = (uint32_t)(((uint64_t)w[k & 3] * (uint64_t)(k + 1)) >> 32);
    uint16_t tmp = perm[k];
    perm[k] = perm[j];
    perm[j] = tmp;
  }
}

void orc_positions(int32_t n, uint32_t w1, uint32_t w2, int32_t *i, int32_t *j) {
  *i = (int32_t)(((uint64_t)w1 * (uint64_t)n) >> 32);
  if (n < 2) {
    *j = *i;
    return;
  }
  int32_t jp = (int32_t)(((uint64_t)w2 * (uint64_t)(n - 1)) >> 32);
  *j = jp + (jp >= *i);
}
