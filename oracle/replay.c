/* Oracle timeline replay -- TEST INFRASTRUCTURE ONLY (see oracle.h).
 *
 * The plain definition of what one priority order costs, simulated one serving
 * iteration at a time:
 *   - all requests are present at time 0 (Algorithm 1 takes the newly arrived jobs);
 *   - requests are admitted in priority order. STATIC: a new batch of up to
 *     max_batch requests starts only when the previous one has drained (batch index
 *     a_i = floor(p_i / B), wait = sum of earlier batch durations, Eqs. for a_i and
 *     t_wait). CONTINUOUS: a finished request frees its slot for the next iteration;
 *   - an admission group costs one prefill iteration equal to the sum of its
 *     members' p0 + p1*l_in; running decodes stall during it. Every admitted request
 *     gets its first token (TTFT) at the end of that iteration;
 *   - each decode iteration costs d0 + d1*b + d2*ctx, b = active requests and ctx =
 *     the sum of their context lengths; the k-th decode step of a request has context
 *     l_in + k (per-token decode model accumulated over l_o tokens);
 *   - a request finishes (e2e) at the end of its l_o-th decode iteration;
 *   - x_i: TTFT <= thr, or e2e <= thr, or TPOT = (e2e - TTFT)/l_o <= thr, the last
 *     checked exactly as e2e - TTFT <= thr * l_o;
 *   - n = sum x_i, t = sum e2e (objective G = n/t, kept as the integer pair).
 */
#include "oracle.h"
#include <stdlib.h>
#include <string.h>

int orc_replay(const orc_queue *q, const orc_model *m, const uint16_t *perm,
               int64_t *n_met, int64_t *t_sum, int64_t *ttft_out, int64_t *e2e_out) {
  const int32_t n = q->n;
  const int32_t B = m->max_batch;
  int32_t *active = (int32_t *)malloc(sizeof(int32_t) * (size_t)(B > n ? n : B) + 4);
  int64_t *gen = (int64_t *)calloc((size_t)n, sizeof(int64_t));
  int64_t *ttft = (int64_t *)calloc((size_t)n, sizeof(int64_t));
  int64_t *e2e = (int64_t *)calloc((size_t)n, sizeof(int64_t));
  char *seen = (char *)calloc((size_t)n, 1);
  int ok = 1;
  for (int32_t p = 0; p < n; p++) {
    if (perm[p] >= n || seen[perm[p]]) { ok = 0; break; }
    seen[perm[p]] = 1;
  }
  if (!ok) {
    free(active); free(gen); free(ttft); free(e2e); free(seen);
    *n_met = -1; *t_sum = -1;
    return -1;
  }

  int64_t t = 0;
  int32_t next = 0, b = 0;
  while (next < n || b > 0) {
    /* both static policies admit a new batch only when the previous one has drained */
    int admit = next < n && (m->policy == ORC_CONTINUOUS ? b < B : b == 0);
    if (admit) {
      int32_t g = B - b;
      if (g > n - next) g = n - next;
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
    for (int32_t u = 0; u < b; u++) {
      int32_t r = active[u];
      ctx += (int64_t)q->in_len[r] + gen[r] + 1;
    }
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
    int met = 0;
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
  free(active); free(gen); free(ttft); free(e2e); free(seen);
  return 0;
}

void orc_eval_rows(const orc_queue *q, const orc_model *m, const uint16_t *perms,
                   int64_t row0, int64_t rows, int64_t *out) {
  for (int64_t k = 0; k < rows; k++) {
    const uint16_t *p = perms + (row0 + k) * (int64_t)q->n;
    orc_replay(q, m, p, &out[2 * k], &out[2 * k + 1], 0, 0);
  }
}

int64_t orc_solo(const orc_queue *q, const orc_model *m, int32_t r) {
  orc_queue one = { 1, &q->in_len[r], &q->out_len[r], &q->kind[r], &q->thr_us[r] };
  uint16_t p = 0;
  int64_t nm, ts;
  orc_replay(&one, m, &p, &nm, &ts, 0, 0);
  return ts;
}
