/* Oracle for the paper's fitted latency predictor -- TEST INFRASTRUCTURE ONLY (see oracle.h).
 *
 * Section "Latency Predictor" taken literally: a request with input length l_i and output
 * length l_o served in a batch of b requests takes
 *   prefill  t_p(b, l_i) = a_p b l_i + b_p b + c_p l_i + d_p                  (eq. for t_p)
 *   decode   t_d = sum over k = 1 .. l_o of tau_d(b, l_i + k),
 *            tau_d(b, l) = a_d b l + b_d b + c_d l + d_d                      (eqs. for tau_d, t_d)
 *   t_exec = t_p + t_d,  TTFT = wait + t_p,  TPOT = t_d / l_o,  e2e = wait + t_exec,
 * with b the size of the request's static batch (constant for the batch, as the per-request
 * model has it). A batch lasts as long as its slowest member (the max in the waiting-time
 * equation) and waits for every earlier batch (Problem Formulation). The coefficients are
 * integers in one time unit chosen by the caller; the paper's Table 2 (milliseconds) is
 * exact in units of 10 ns. The decode sum is taken term by term here.
 *
 * SLO kinds: TTFT, TPOT or end-to-end as before, and kind 3, the paper's chat SLO (h_i = 0
 * in the definition of x_i): TTFT <= thr AND TPOT <= thr2, with thr2 from a second
 * per-request array. TPOT is checked exactly as t_d <= thr * l_o.
 */
#include "oracle.h"
#include <stdlib.h>
#include <string.h>

int64_t orc_fit_prefill(const orc_fit_model *f, int64_t b, int64_t l) {
  return f->ap * b * l + f->bp * b + f->cp * l + f->dp;
}

int64_t orc_fit_decode(const orc_fit_model *f, int64_t b, int64_t l, int64_t L) {
  int64_t t = 0;
  for (int64_t k = 1; k <= L; k++) t += f->ad * b * (l + k) + f->bd * b + f->cd * (l + k) + f->dd;
  return t;
}

static int met_fit(uint8_t kind, int64_t thr, int64_t thr2, int64_t L, int64_t ttft, int64_t td, int64_t e2e) {
  if (kind == ORC_TTFT) return ttft <= thr;
  if (kind == ORC_E2E) return e2e <= thr;
  if (kind == ORC_TPOT) return td <= thr * L;
  return ttft <= thr && td <= thr2 * L; /* ORC_TTFT_TPOT */
}

int orc_replay_fit(const orc_queue *q, const orc_fit_model *f, const uint16_t *perm, const uint8_t *starts,
                   const uint32_t *thr2, int64_t *n_met, int64_t *t_sum, int64_t *ttft_out, int64_t *e2e_out) {
  const int32_t n = q->n;
  uint8_t *st = (uint8_t *)malloc((size_t)n);
  if (starts) memcpy(st, starts, (size_t)n);
  else orc_max_starts(n, f->max_batch, st);
  char *seen = (char *)calloc((size_t)n, 1);
  int ok = orc_check_starts(st, n, f->max_batch);
  for (int32_t p = 0; ok && p < n; p++) {
    if (perm[p] >= n || seen[perm[p]] || q->kind[perm[p]] > 3 || (q->kind[perm[p]] == 3 && !thr2)) ok = 0;
    else seen[perm[p]] = 1;
  }
  free(seen);
  if (!ok) {
    free(st);
    *n_met = -1;
    *t_sum = -1;
    return -1;
  }
  int64_t wait = 0, nm = 0, ts = 0;
  for (int32_t s = 0; s < n;) {
    int32_t e = s + 1;
    while (e < n && !st[e]) e++;
    const int64_t b = e - s;
    int64_t dur = 0;
    for (int32_t p = s; p < e; p++) {
      const int32_t r = perm[p];
      const int64_t l = q->in_len[r], L = q->out_len[r];
      const int64_t tp = orc_fit_prefill(f, b, l), td = orc_fit_decode(f, b, l, L);
      const int64_t ttft = wait + tp, e2e = wait + tp + td;
      if (tp + td > dur) dur = tp + td;
      nm += met_fit(q->kind[r], q->thr_us[r], thr2 ? thr2[r] : 0, L, ttft, td, e2e);
      ts += e2e;
      if (ttft_out) ttft_out[r] = ttft;
      if (e2e_out) e2e_out[r] = e2e;
    }
    wait += dur;
    s = e;
  }
  free(st);
  *n_met = nm;
  *t_sum = ts;
  return 0;
}

int orc_start_fit(const orc_queue *q, const orc_fit_model *f, const orc_search *s, const uint32_t *thr2,
                  uint16_t *start, int64_t *t_ref, int64_t *start_n, int64_t *start_t) {
  const int32_t n = q->n;
  int64_t *solo = (int64_t *)malloc(sizeof(int64_t) * (size_t)n);
  /* predicted latency of a request served alone (batch of one), the sort key of Algorithm 1 */
  for (int32_t r = 0; r < n; r++)
    solo[r] = orc_fit_prefill(f, 1, q->in_len[r]) + orc_fit_decode(f, 1, q->in_len[r], q->out_len[r]);
  for (int32_t p = 0; p < n; p++) {
    int32_t u = p;
    while (u > 0 && solo[start[u - 1]] > solo[p]) {
      start[u] = start[u - 1];
      u--;
    }
    start[u] = (uint16_t)p;
  }
  int64_t sn, stt, in_n, in_t;
  orc_replay_fit(q, f, start, 0, thr2, &sn, &stt, 0, 0);
  const int allmet = sn == n;
  uint16_t *ident = (uint16_t *)malloc(sizeof(uint16_t) * (size_t)n);
  for (int32_t p = 0; p < n; p++) ident[p] = (uint16_t)p;
  orc_replay_fit(q, f, ident, 0, thr2, &in_n, &in_t, 0, 0);
  if (!(s->early_exit && allmet) && orc_better(s, in_n, in_t, sn, stt)) {
    memcpy(start, ident, sizeof(uint16_t) * (size_t)n);
    sn = in_n;
    stt = in_t;
  }
  *t_ref = f->t_ref > 0 ? f->t_ref : (in_t > 1 ? in_t : 1);
  *start_n = sn;
  *start_t = stt;
  free(solo);
  free(ident);
  return allmet;
}

#define FNV_OFFSET 0xCBF29CE484222325ull
#define FNV_PRIME 0x100000001B3ull

void orc_anneal_chain_fit(const orc_queue *q, const orc_fit_model *f, const orc_search *s, const uint32_t *thr2,
                          const uint16_t *start, int64_t t_ref, int allmet, int32_t chain, int32_t iters, double T0,
                          double alpha, uint64_t seed, uint16_t *cur, uint8_t *cur_starts, uint16_t *best,
                          uint8_t *best_starts, int64_t *rec) {
  const int32_t n = q->n, B = f->max_batch;
  const int search = f->policy == ORC_STATIC_SEARCH;
  uint16_t *cand = (uint16_t *)malloc(sizeof(uint16_t) * (size_t)n);
  uint8_t *cst = (uint8_t *)malloc((size_t)n);
  memcpy(cur, start, sizeof(uint16_t) * (size_t)n);
  orc_max_starts(n, B, cur_starts);
  memcpy(best, cur, sizeof(uint16_t) * (size_t)n);
  memcpy(best_starts, cur_starts, (size_t)n);
  int64_t cn, ct;
  orc_replay_fit(q, f, cur, cur_starts, thr2, &cn, &ct, 0, 0);
  int64_t bn = cn, bt = ct, biter = -1, accepts = 0;
  uint64_t digest = FNV_OFFSET;
  uint32_t key[2] = { (uint32_t)seed, (uint32_t)(seed >> 32) };
  if (s->early_exit && allmet) iters = 0;
  int32_t level_left = s->level_len;
  double T = T0;
  for (int32_t k = 0; k < iters; k++) {
    uint32_t ctr[4] = { (uint32_t)k, (uint32_t)chain, 0u, (uint32_t)ORC_TAG_ANNEAL };
    uint32_t w[4];
    orc_philox(ctr, key, w);
    int32_t i, j;
    orc_positions(n, w[1], w[2], &i, &j);
    memcpy(cand, cur, sizeof(uint16_t) * (size_t)n);
    memcpy(cst, cur_starts, (size_t)n);
    int made = 1;
    if (search) {
      const int op = orc_op3(w[0]);
      if (op == 0) made = orc_squeeze(cand, cst, n, B, i);
      else if (op == 1) made = orc_delay(cand, cst, n, B, i);
      else if (n >= 2) orc_swap(cand, i, j);
      else made = 0;
    } else {
      if ((uint64_t)w[0] < f->swap_threshold) orc_swap(cand, i, j);
      else orc_insert(cand, i, j);
    }
    if (made) {
      int64_t nn, nt;
      orc_replay_fit(q, f, cand, cst, thr2, &nn, &nt, 0, 0);
      int acc;
      if (s->objective == ORC_OBJ_RATIO) {
        acc = orc_accept_ratio(nn * ct - cn * nt, t_ref, ct, nt, T, w[3]);
      } else {
        acc = orc_accept((nn - cn) * t_ref - (nt - ct), t_ref, T, w[3]);
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
