/* Oracle for the joint search over priority order and batch sizes -- TEST INFRASTRUCTURE
 * ONLY (see oracle.h).
 *
 * Problem Formulation: the batch sizes are a sequence b_0 .. b_{M-1} with sum N, each at
 * most the preset maximum, and a job at position p belongs to the batch whose cumulated
 * sizes bracket p; the argmax runs over the order AND the batch indices. Here the sizes
 * are carried as one start flag per position (1 where a batch begins; position 0 always
 * begins one), and a batch runs until the next flag.
 *
 * Algorithm 1 and the section "Priority Mapping Algorithm" give three ways to make a new
 * solution, picked uniformly:
 *   - squeezeLastIter: move a request into the previous batch (the one that runs just
 *     before its own), allowed when it is not in the first batch and that batch is below
 *     the maximum size;
 *   - delayNextIter: move a request into the next batch, allowed when that batch is below
 *     the maximum size. For the last batch, the next batch is a new one, opened only when
 *     the request does not run alone (otherwise nothing would change);
 *   - randSwapping: exchange two positions of the order (batch sizes unchanged).
 * A moved request takes the adjoining end of its new batch: the last position of the
 * previous batch (squeeze) or the first position of the next one (delay); members of a
 * static batch start together, so their order inside the batch does not change any
 * latency. A move that is not allowed leaves the solution unchanged and counts as neither
 * accepted nor rejected. Start solutions use the maximum batch size everywhere, as the
 * paper's input-order start does.
 */
#include "oracle.h"
#include <stdlib.h>
#include <string.h>

static int better_key(int64_t n1, int64_t t1, int64_t n2, int64_t t2) {
  return n1 > n2 || (n1 == n2 && t1 < t2);
}

int orc_check_starts(const uint8_t *starts, int32_t n, int32_t B) {
  if (n < 1 || starts[0] != 1) return 0;
  int32_t run = 0;
  for (int32_t p = 0; p < n; p++) {
    if (starts[p] > 1) return 0;
    run = starts[p] ? 1 : run + 1;
    if (run > B) return 0;
  }
  return 1;
}

void orc_max_starts(int32_t n, int32_t B, uint8_t *starts) {
  for (int32_t p = 0; p < n; p++) starts[p] = (uint8_t)(p % B == 0);
}

int orc_replay_batches(const orc_queue *q, const orc_model *m, const uint16_t *perm,
                       const uint8_t *starts, int64_t *n_met, int64_t *t_sum, int64_t *ttft_out,
                       int64_t *e2e_out) {
  const int32_t n = q->n;
  char *seen = (char *)calloc((size_t)n, 1);
  int ok = orc_check_starts(starts, n, m->max_batch);
  for (int32_t p = 0; ok && p < n; p++) {
    if (perm[p] >= n || seen[perm[p]]) ok = 0;
    else seen[perm[p]] = 1;
  }
  free(seen);
  if (!ok) {
    *n_met = -1;
    *t_sum = -1;
    return -1;
  }
  int32_t *active = (int32_t *)malloc(sizeof(int32_t) * (size_t)n);
  int64_t *gen = (int64_t *)calloc((size_t)n, sizeof(int64_t));
  int64_t *ttft = (int64_t *)calloc((size_t)n, sizeof(int64_t));
  int64_t *e2e = (int64_t *)calloc((size_t)n, sizeof(int64_t));

  /* one serving iteration at a time: a batch is admitted when the previous one has
   * drained; its prefill is one iteration; then decode iterations until it drains */
  int64_t t = 0;
  int32_t next = 0, b = 0;
  while (next < n || b > 0) {
    if (b == 0) {
      int32_t g = 1;
      while (next + g < n && !starts[next + g]) g++;
      int64_t pre = 0;
      for (int32_t u = 0; u < g; u++) pre += m->p0 + m->p1 * (int64_t)q->in_len[perm[next + u]];
      t += pre;
      for (int32_t u = 0; u < g; u++) {
        int32_t r = perm[next + u];
        ttft[r] = t;
        active[b++] = r;
      }
      next += g;
    }
    int64_t ctx = 0;
    for (int32_t u = 0; u < b; u++) ctx += (int64_t)q->in_len[active[u]] + gen[active[u]] + 1;
    t += m->d0 + m->d1 * (int64_t)b + m->d2 * ctx;
    int32_t keep = 0;
    for (int32_t u = 0; u < b; u++) {
      int32_t r = active[u];
      gen[r] += 1;
      if (gen[r] == (int64_t)q->out_len[r]) e2e[r] = t;
      else active[keep++] = r;
    }
    b = keep;
  }

  int64_t nm = 0, ts = 0;
  for (int32_t r = 0; r < n; r++) {
    int met;
    if (q->kind[r] == ORC_TTFT) met = ttft[r] <= (int64_t)q->thr_us[r];
    else if (q->kind[r] == ORC_E2E) met = e2e[r] <= (int64_t)q->thr_us[r];
    else met = e2e[r] - ttft[r] <= (int64_t)q->thr_us[r] * (int64_t)q->out_len[r];
    nm += met;
    ts += e2e[r];
  }
  *n_met = nm;
  *t_sum = ts;
  if (ttft_out) memcpy(ttft_out, ttft, sizeof(int64_t) * (size_t)n);
  if (e2e_out) memcpy(e2e_out, e2e, sizeof(int64_t) * (size_t)n);
  free(active); free(gen); free(ttft); free(e2e);
  return 0;
}

void orc_eval_rows_batches(const orc_queue *q, const orc_model *m, const uint16_t *perms,
                           const uint8_t *starts, int64_t row0, int64_t rows, int64_t *out) {
  for (int64_t k = 0; k < rows; k++) {
    const int64_t off = (row0 + k) * (int64_t)q->n;
    orc_replay_batches(q, m, perms + off, starts + off, &out[2 * k], &out[2 * k + 1], 0, 0);
  }
}

/* first position of the batch holding p, and the first position after it */
static void batch_bounds(const uint8_t *starts, int32_t n, int32_t p, int32_t *s, int32_t *e) {
  int32_t a = p, z = p + 1;
  while (!starts[a]) a--;
  while (z < n && !starts[z]) z++;
  *s = a;
  *e = z;
}

int orc_squeeze(uint16_t *perm, uint8_t *starts, int32_t n, int32_t B, int32_t i) {
  int32_t s, e, sp, ep;
  batch_bounds(starts, n, i, &s, &e);
  if (s == 0) return 0;                 /* already in the first batch */
  batch_bounds(starts, n, s - 1, &sp, &ep);
  if (s - sp >= B) return 0;            /* previous batch is full */
  orc_insert(perm, i, s);               /* becomes the previous batch's last member */
  starts[s] = 0;
  if (s + 1 < e) starts[s + 1] = 1;     /* the rest of its old batch, if any, starts after it */
  return 1;
}

int orc_delay(uint16_t *perm, uint8_t *starts, int32_t n, int32_t B, int32_t i) {
  int32_t s, e, sn, en;
  batch_bounds(starts, n, i, &s, &e);
  if (e == n) {
    if (e - s < 2) return 0;            /* alone in the last batch: nothing to split off */
    orc_insert(perm, i, e - 1);         /* opens a new last batch */
    starts[e - 1] = 1;
    return 1;
  }
  batch_bounds(starts, n, e, &sn, &en);
  if (en - sn >= B) return 0;           /* next batch is full */
  orc_insert(perm, i, e - 1);           /* becomes the next batch's first member */
  starts[e] = 0;
  starts[e - 1] = 1;
  return 1;
}

int orc_op3(uint32_t w0) { return (int)(((uint64_t)w0 * 3u) >> 32); }

#define FNV_OFFSET 0xCBF29CE484222325ull
#define FNV_PRIME 0x100000001B3ull

void orc_anneal_chain_batches(const orc_queue *q, const orc_model *m, const uint16_t *start,
                              int64_t t_ref, int allmet, int32_t chain, int32_t iters, double T0,
                              double alpha, uint64_t seed, uint16_t *cur, uint8_t *cur_starts,
                              uint16_t *best, uint8_t *best_starts, int64_t *rec, int64_t *trace) {
  const orc_search lex = { ORC_OBJ_LEX, 1, 0, 0 };
  orc_anneal_chain_batches_ex(q, m, &lex, start, t_ref, allmet, chain, iters, T0, alpha, seed, cur,
                              cur_starts, best, best_starts, rec, trace);
}

void orc_anneal_chain_batches_ex(const orc_queue *q, const orc_model *m, const orc_search *s,
                                 const uint16_t *start, int64_t t_ref, int allmet, int32_t chain,
                                 int32_t iters, double T0, double alpha, uint64_t seed,
                                 uint16_t *cur, uint8_t *cur_starts, uint16_t *best,
                                 uint8_t *best_starts, int64_t *rec, int64_t *trace) {
  const int32_t n = q->n, B = m->max_batch;
  if (s->early_exit && allmet) iters = 0;
  int32_t level_left = s->level_len;
  uint16_t *cand = (uint16_t *)malloc(sizeof(uint16_t) * (size_t)n);
  uint8_t *cst = (uint8_t *)malloc((size_t)n);
  memcpy(cur, start, sizeof(uint16_t) * (size_t)n);
  orc_max_starts(n, B, cur_starts);
  memcpy(best, cur, sizeof(uint16_t) * (size_t)n);
  memcpy(best_starts, cur_starts, (size_t)n);
  int64_t cn, ct;
  orc_replay_batches(q, m, cur, cur_starts, &cn, &ct, 0, 0);
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
    int op = orc_op3(w[0]);
    memcpy(cand, cur, sizeof(uint16_t) * (size_t)n);
    memcpy(cst, cur_starts, (size_t)n);
    int made;
    if (op == 0) made = orc_squeeze(cand, cst, n, B, i);
    else if (op == 1) made = orc_delay(cand, cst, n, B, i);
    else {
      made = n >= 2;
      if (made) orc_swap(cand, i, j);
    }
    int acc = 0;
    if (made) {
      int64_t nn, nt;
      orc_replay_batches(q, m, cand, cst, &nn, &nt, 0, 0);
      if (s->objective == ORC_OBJ_RATIO) {
        acc = orc_accept_ratio(nn * ct - cn * nt, t_ref, ct, nt, T, w[3]);
      } else {
        int64_t delta = (nn - cn) * t_ref - (nt - ct);
        acc = orc_accept(delta, t_ref, T, w[3]);
      }
      if (acc) {
        memcpy(cur, cand, sizeof(uint16_t) * (size_t)n);
        memcpy(cur_starts, cst, (size_t)n);
        cn = nn;
        ct = nt;
        accepts++;
        if (orc_better(s, cn, ct, bn, bt)) {
          memcpy(best, cur, sizeof(uint16_t) * (size_t)n);
          memcpy(best_starts, cur_starts, (size_t)n);
          bn = cn;
          bt = ct;
          biter = k;
        }
        digest = (digest ^ (uint64_t)k) * FNV_PRIME;
        digest = (digest ^ (uint64_t)cn) * FNV_PRIME;
        digest = (digest ^ (uint64_t)ct) * FNV_PRIME;
      }
    }
    if (trace) {
      trace[4 * (int64_t)k + 0] = acc;
      trace[4 * (int64_t)k + 1] = cn;
      trace[4 * (int64_t)k + 2] = ct;
      trace[4 * (int64_t)k + 3] = op | (made ? 0 : 4);
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
  free(cst);
}

/* lexicographic successor; returns 0 after the last permutation */
static int next_order(uint16_t *p, int32_t n) {
  int32_t i = n - 2;
  while (i >= 0 && p[i] >= p[i + 1]) i--;
  if (i < 0) return 0;
  int32_t j = n - 1;
  while (p[j] <= p[i]) j--;
  orc_swap(p, i, j);
  for (int32_t a = i + 1, b = n - 1; a < b; a++, b--) orc_swap(p, a, b);
  return 1;
}

int64_t orc_brute_batches(const orc_queue *q, const orc_model *m, int64_t *best_n, int64_t *best_t,
                          uint16_t *best_perm, uint8_t *best_starts) {
  const int32_t n = q->n;
  uint16_t p[16];
  uint8_t st[16];
  for (int32_t u = 0; u < n; u++) p[u] = (uint16_t)u;
  int64_t bn = -1, bt = 0, count = 0;
  do {
    /* bit u-1 of mask set <=> a batch starts at position u (u = 1 .. n-1) */
    for (uint32_t mask = 0; mask < (1u << (n - 1)); mask++) {
      st[0] = 1;
      for (int32_t u = 1; u < n; u++) st[u] = (uint8_t)((mask >> (u - 1)) & 1u);
      if (!orc_check_starts(st, n, m->max_batch)) continue;
      int64_t nn, nt;
      orc_replay_batches(q, m, p, st, &nn, &nt, 0, 0);
      if (bn < 0 || better_key(nn, nt, bn, bt)) {
        bn = nn;
        bt = nt;
        count = 1;
        memcpy(best_perm, p, sizeof(uint16_t) * (size_t)n);
        memcpy(best_starts, st, (size_t)n);
      } else if (nn == bn && nt == bt) {
        count++;
      }
    }
  } while (next_order(p, n));
  *best_n = bn;
  *best_t = bt;
  return count;
}
