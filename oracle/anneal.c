/* Oracle annealing chain, start order and exhaustive search -- TEST INFRASTRUCTURE ONLY
 * (see oracle.h).
 *
 * Follows Algorithm 1 ("Simulated-Annealing Priority Mapping") with these readings:
 *   - start: sort the jobs by their predicted solo end-to-end latency (stable, ties by
 *     index); the input order replaces it if its key is strictly better. The early
 *     exit when the sorted order meets every SLO is reported as a flag only;
 *   - one proposal per iteration, cooled geometrically: T_k = T0 * alpha^k, formed by
 *     one fp64 multiply per iteration; with search settings, one multiply per level of
 *     level_len proposals (T_k = T0 * alpha^floor(k / level_len)), the paper's per-level
 *     cooling;
 *   - proposals: swap two positions (randSwapping) or remove one request and re-insert
 *     it elsewhere; batches are formed by the admission policy. The joint search over
 *     order and batch sizes with the paper's squeeze / delay moves is in sized.c;
 *   - acceptance: see orc_accept (rng.c); equal scores are accepted;
 *   - score order: (n1, t1) beats (n2, t2) iff n1 > n2, or n1 == n2 and t1 < t2
 *     (attainment first, then mean latency); with the ratio objective iff n1 t2 > n2 t1
 *     (G = n / t of the Problem Formulation), accepted by orc_accept_ratio;
 *   - every chain also keeps its best-so-far order (strict improvements only).
 * Random draws: one Philox4x32-10 block per (seed, chain, iteration), counter
 * (iteration, chain, 0, ORC_TAG_ANNEAL), key (seed low, seed high). Word 0 picks the
 * move (swap iff w0 < swap_threshold), words 1 and 2 the positions, word 3 the uniform
 * u = w3 * 2^-32 of the acceptance test.
 */
#include "oracle.h"
#include <stdlib.h>
#include <string.h>

void orc_swap(uint16_t *p, int32_t i, int32_t j) {
  uint16_t t = p[i];
  p[i] = p[j];
  p[j] = t;
}

void orc_insert(uint16_t *p, int32_t from, int32_t to) {
  uint16_t x = p[from];
  if (from < to) {
    for (int32_t u = from; u < to; u++) p[u] = p[u + 1];
  } else {
    for (int32_t u = from; u > to; u--) p[u] = p[u - 1];
  }
  p[to] = x;
}

static const orc_search DEFAULT_SEARCH = { ORC_OBJ_LEX, 1, 0, 0 };

int orc_better(const orc_search *s, int64_t n1, int64_t t1, int64_t n2, int64_t t2) {
  if (s->objective == ORC_OBJ_RATIO) return n1 * t2 > n2 * t1;
  return n1 > n2 || (n1 == n2 && t1 < t2);
}

int orc_start(const orc_queue *q, const orc_model *m, uint16_t *start, int64_t *t_ref,
              int64_t *start_n, int64_t *start_t) {
  return orc_start_ex(q, m, &DEFAULT_SEARCH, start, t_ref, start_n, start_t);
}

int orc_start_ex(const orc_queue *q, const orc_model *m, const orc_search *s, uint16_t *start,
                 int64_t *t_ref, int64_t *start_n, int64_t *start_t) {
  const int32_t n = q->n;
  int64_t *solo = (int64_t *)malloc(sizeof(int64_t) * (size_t)n);
  for (int32_t r = 0; r < n; r++) solo[r] = orc_solo(q, m, r);
  /* stable insertion sort of request ids by solo latency */
  for (int32_t p = 0; p < n; p++) {
    int32_t u = p;
    while (u > 0 && solo[start[u - 1]] > solo[p]) {
      start[u] = start[u - 1];
      u--;
    }
    start[u] = (uint16_t)p;
  }
  int64_t sn, st, in_n, in_t;
  orc_replay(q, m, start, &sn, &st, 0, 0);
  int allmet = sn == n;
  uint16_t *ident = (uint16_t *)malloc(sizeof(uint16_t) * (size_t)n);
  for (int32_t p = 0; p < n; p++) ident[p] = (uint16_t)p;
  orc_replay(q, m, ident, &in_n, &in_t, 0, 0);
  /* the early exit keeps the sorted order; otherwise the better of the two starts */
  if (!(s->early_exit && allmet) && orc_better(s, in_n, in_t, sn, st)) {
    memcpy(start, ident, sizeof(uint16_t) * (size_t)n);
    sn = in_n;
    st = in_t;
  }
  *t_ref = m->t_ref_us > 0 ? m->t_ref_us : (in_t > 1 ? in_t : 1);
  *start_n = sn;
  *start_t = st;
  free(solo);
  free(ident);
  return allmet;
}

#define FNV_OFFSET 0xCBF29CE484222325ull
#define FNV_PRIME 0x100000001B3ull

void orc_anneal_chain(const orc_queue *q, const orc_model *m, const uint16_t *start,
                      int64_t t_ref, int allmet, int32_t chain, int32_t iters, double T0,
                      double alpha, uint64_t seed, uint16_t *cur, uint16_t *best, int64_t *rec,
                      int64_t *trace) {
  orc_anneal_chain_ex(q, m, &DEFAULT_SEARCH, start, t_ref, allmet, chain, iters, T0, alpha, seed,
                      cur, best, rec, trace);
}

void orc_anneal_chain_ex(const orc_queue *q, const orc_model *m, const orc_search *s,
                         const uint16_t *start, int64_t t_ref, int allmet, int32_t chain,
                         int32_t iters, double T0, double alpha, uint64_t seed, uint16_t *cur,
                         uint16_t *best, int64_t *rec, int64_t *trace) {
  const int32_t n = q->n;
  if (s->early_exit && allmet) iters = 0;
  int32_t level_left = s->level_len;
  uint16_t *cand = (uint16_t *)malloc(sizeof(uint16_t) * (size_t)n);
  memcpy(cur, start, sizeof(uint16_t) * (size_t)n);
  memcpy(best, start, sizeof(uint16_t) * (size_t)n);
  int64_t cn, ct;
  orc_replay(q, m, cur, &cn, &ct, 0, 0);
  int64_t bn = cn, bt = ct, biter = -1, accepts = 0;
  uint64_t digest = FNV_OFFSET;
  uint32_t key[2] = { (uint32_t)seed, (uint32_t)(seed >> 32) };
  double T = T0;
  for (int32_t k = 0; k < iters; k++) {
    uint32_t ctr[4] = { (uint32_t)k, (uint32_t)chain, 0u, (uint32_t)ORC_TAG_ANNEAL };
    uint32_t w[4];
    orc_philox(ctr, key, w);
    int32_t i, j;
    orc_positions(n, w[1], w[2], &i, &j);
    int move = (uint64_t)w[0] < m->swap_threshold ? 0 : 1;
    memcpy(cand, cur, sizeof(uint16_t) * (size_t)n);
    if (move == 0) orc_swap(cand, i, j);
    else orc_insert(cand, i, j);
    int64_t nn, nt;
    orc_replay(q, m, cand, &nn, &nt, 0, 0);
    int acc;
    if (s->objective == ORC_OBJ_RATIO) {
      acc = orc_accept_ratio(nn * ct - cn * nt, t_ref, ct, nt, T, w[3]);
    } else {
      int64_t delta = (nn - cn) * t_ref - (nt - ct);
      acc = orc_accept(delta, t_ref, T, w[3]);
    }
    if (acc) {
      memcpy(cur, cand, sizeof(uint16_t) * (size_t)n);
      cn = nn;
      ct = nt;
      accepts++;
      if (orc_better(s, cn, ct, bn, bt)) {
        memcpy(best, cur, sizeof(uint16_t) * (size_t)n);
        bn = cn;
        bt = ct;
        biter = k;
      }
      digest = (digest ^ (uint64_t)k) * FNV_PRIME;
      digest = (digest ^ (uint64_t)cn) * FNV_PRIME;
      digest = (digest ^ (uint64_t)ct) * FNV_PRIME;
    }
    if (trace) {
      trace[4 * (int64_t)k + 0] = acc;
      trace[4 * (int64_t)k + 1] = cn;
      trace[4 * (int64_t)k + 2] = ct;
      trace[4 * (int64_t)k + 3] = move;
    }
    if (--level_left == 0) {
      level_left = s->level_len;
      T = T * alpha;
    }
  }
  rec[ORC_R_CUR_N] = cn;
  rec[ORC_R_CUR_T] = ct;
  rec[ORC_R_BEST_N] = bn;
  rec[ORC_R_BEST_T] = bt;
  rec[ORC_R_BEST_ITER] = biter;
  rec[ORC_R_ACCEPTS] = accepts;
  rec[ORC_R_DIGEST] = (int64_t)digest;
  rec[ORC_R_ALLMET] = allmet;
  free(cand);
}

/* lexicographic successor; returns 0 after the last permutation */
static int next_perm(uint16_t *p, int32_t n) {
  int32_t i = n - 2;
  while (i >= 0 && p[i] >= p[i + 1]) i--;
  if (i < 0) return 0;
  int32_t j = n - 1;
  while (p[j] <= p[i]) j--;
  orc_swap(p, i, j);
  for (int32_t a = i + 1, b = n - 1; a < b; a++, b--) orc_swap(p, a, b);
  return 1;
}

int64_t orc_brute(const orc_queue *q, const orc_model *m, int64_t *best_n, int64_t *best_t,
                  uint16_t *best_perm) {
  return orc_brute_ex(q, m, &DEFAULT_SEARCH, best_n, best_t, best_perm);
}

int64_t orc_brute_ex(const orc_queue *q, const orc_model *m, const orc_search *s, int64_t *best_n,
                     int64_t *best_t, uint16_t *best_perm) {
  const int32_t n = q->n;
  uint16_t p[16];
  for (int32_t u = 0; u < n; u++) p[u] = (uint16_t)u;
  int64_t bn = -1, bt = 0, count = 0;
  do {
    int64_t nn, nt;
    orc_replay(q, m, p, &nn, &nt, 0, 0);
    if (bn < 0 || orc_better(s, nn, nt, bn, bt)) {
      bn = nn;
      bt = nt;
      count = 1;
      memcpy(best_perm, p, sizeof(uint16_t) * (size_t)n);
    } else if (!orc_better(s, bn, bt, nn, nt)) {
      count++;  /* as good as the best: equal key, or equal ratio */
    }
  } while (next_perm(p, n));
  *best_n = bn;
  *best_t = bt;
  return count;
}
