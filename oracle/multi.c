/* Oracle for the multi-instance scheduling solution -- TEST INFRASTRUCTURE ONLY (see
 * oracle.h).
 *
 * Section "Scheduling Solution", instance assignment (Algorithm 2's InstAssign): requests
 * are taken in arrival order and each goes to the instance with the largest remaining
 * memory, expressed in tokens (token_num(m) = m * mu / sigma, computed by the caller as
 * each instance's capacity). When even that instance cannot hold the request, every
 * instance's remaining memory is reset to its capacity -- a fresh iteration starts -- and
 * the request goes to the instance with the largest capacity. Readings: a request holds
 * l_in + l_out tokens (prompt and predicted output); ties go to the lowest instance index;
 * after a reset the request is placed even if it exceeds the capacity (the next request
 * then starts another iteration). Each instance then orders its own requests
 * independently (priority mapping within each instance), which the tests compose from
 * orc_start and orc_anneal_chain on the instance's requests in arrival order.
 */
#include "oracle.h"

void orc_assign(const orc_queue *q, int32_t instances, const int64_t *capacity, int32_t *inst_out) {
  int64_t rem[64];
  for (int32_t k = 0; k < instances; k++) rem[k] = capacity[k];
  for (int32_t r = 0; r < q->n; r++) {
    const int64_t need = (int64_t)q->in_len[r] + (int64_t)q->out_len[r];
    int32_t best = 0;
    for (int32_t k = 1; k < instances; k++)
      if (rem[k] > rem[best]) best = k;
    if (rem[best] < need) {
      for (int32_t k = 0; k < instances; k++) rem[k] = capacity[k];
      best = 0;
      for (int32_t k = 1; k < instances; k++)
        if (rem[k] > rem[best]) best = k;
    }
    rem[best] -= need;
    inst_out[r] = best;
  }
}
