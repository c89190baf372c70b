/* CPU oracle for the SLO-aware simulated-annealing scheduler -- TEST INFRASTRUCTURE ONLY.
 *
 * Plain, slow, single-threaded C. Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg may call it. It shares no code, header, table or
 * constant with the GPU library; the two meet only through the seeded input
 * generator and through the results the tests compare.
 *
 * Paper: "SLO-Aware Scheduling for Large Language Model Inferences" (Huang et al.).
 *   - objective and SLO flags: Section "Problem Formulation", Eqs. for G = n/t,
 *     t = sum of e2e latencies, n = sum x_i, x_i, TTFT, TPOT;
 *   - latency model: Section "Latency Predictor" (prefill, per-token decode and its
 *     accumulation over the output tokens, TPOT = decode time / output length);
 *   - search: Algorithm 1 "Simulated-Annealing Priority Mapping" and Section
 *     "Priority Mapping Algorithm".
 *
 * All latencies are int64 microseconds. The only floating point is the fp64
 * Metropolis test (orc_accept), compiled without FMA contraction or fast-math.
 *
 * Parity pins (what checks this oracle against something other than itself) are
 * listed per function below; "parity unpinned" marks the annealing trajectory,
 * which has no published values and is checked only for its properties.
 */
#ifndef SLO_ORACLE_H
#define SLO_ORACLE_H
#include <stdint.h>

enum { ORC_TTFT = 0, ORC_TPOT = 1, ORC_E2E = 2 };
/* ORC_STATIC_SEARCH: static admission whose batch sizes are searched together with the
 * order (batch-size sequence of the Problem Formulation, squeeze / delay moves of
 * Algorithm 1). Replayed with maximum-size batches it is ORC_STATIC. */
enum { ORC_STATIC = 0, ORC_CONTINUOUS = 1, ORC_STATIC_SEARCH = 2 };
enum { ORC_TAG_ANNEAL = 0x53414e4e, ORC_TAG_FY = 0x46495348 };

typedef struct {
  int32_t n;
  const uint16_t *in_len, *out_len;
  const uint8_t *kind;
  const uint32_t *thr_us;
} orc_queue;

typedef struct {
  int32_t max_batch, policy;
  int64_t p0, p1, d0, d1, d2;
  int64_t t_ref_us;
  uint64_t swap_threshold;
} orc_model;

/* per-chain record layout (int64 each) */
enum { ORC_R_CUR_N, ORC_R_CUR_T, ORC_R_BEST_N, ORC_R_BEST_T, ORC_R_BEST_ITER,
       ORC_R_ACCEPTS, ORC_R_DIGEST, ORC_R_ALLMET, ORC_R_WORDS };

/* Step-by-step timeline of one priority order. Returns 0, or -1 if perm is not a
 * permutation of 0..n-1. ttft/e2e (nullable) receive per-request values indexed by
 * request id. Pinned by hand-worked timelines, Smith's rule at batch size 1,
 * closed-form decode sums, and batching invariants. */
int orc_replay(const orc_queue *q, const orc_model *m, const uint16_t *perm,
               int64_t *n_met, int64_t *t_sum, int64_t *ttft, int64_t *e2e);

/* Rows of a k x n permutation matrix; out is k x 2 (n_met, t_sum) or (-1,-1). */
void orc_eval_rows(const orc_queue *q, const orc_model *m, const uint16_t *perms,
                   int64_t row0, int64_t rows, int64_t *out);

/* Philox4x32-10 block (Salmon et al., SC'11). Pinned by published known-answer vectors. */
void orc_philox(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4]);

/* exp(x) for x <= 0 by Cody-Waite reduction and a Taylor polynomial; 0 below -708.
 * Pinned by its error against the C library exp. */
double orc_det_exp(double x);

/* Metropolis acceptance for a maximisation with energy f = n - t/t_ref:
 * accept iff delta >= 0, or u < exp(delta / (t_ref * T)) with u = w3 * 2^-32. */
int orc_accept(int64_t delta, int64_t t_ref, double T, uint32_t w3);

/* Fisher-Yates shuffle of 0..n-1, draws from Philox keyed by seed, row idx. */
void orc_fy_perm(uint64_t seed, int32_t n, uint32_t idx, uint16_t *perm);

/* Start of every chain (Algorithm 1 initialisation): stable sort by solo latency;
 * the input order replaces it when its key is strictly better. Returns allmet flag. */
int orc_start(const orc_queue *q, const orc_model *m, uint16_t *start, int64_t *t_ref,
              int64_t *start_n, int64_t *start_t);

/* The two moves. */
void orc_swap(uint16_t *p, int32_t i, int32_t j);
void orc_insert(uint16_t *p, int32_t from, int32_t to);

/* Proposal positions from one Philox block (i uniform, j uniform over the others). */
void orc_positions(int32_t n, uint32_t w1, uint32_t w2, int32_t *i, int32_t *j);

/* One annealing chain. start/t_ref from orc_start. cur/best receive n entries,
 * rec ORC_R_WORDS int64. trace (nullable) receives iters x 4 int64:
 * (accepted, n, t, move) after each proposal. Parity unpinned (trajectory). */
void orc_anneal_chain(const orc_queue *q, const orc_model *m, const uint16_t *start,
                      int64_t t_ref, int allmet, int32_t chain, int32_t iters, double T0,
                      double alpha, uint64_t seed, uint16_t *cur, uint16_t *best, int64_t *rec,
                      int64_t *trace);

/* Exhaustive search over all n! orders (n <= 10): optimum key and the
 * lexicographically first optimal order; returns the number of optimal orders. */
int64_t orc_brute(const orc_queue *q, const orc_model *m, int64_t *best_n, int64_t *best_t,
                  uint16_t *best_perm);

/* ---- the paper's own schedule and objective (search settings) ----
 * objective ORC_OBJ_LEX: attainment first, then lower total latency (energy n - t/t_ref).
 * objective ORC_OBJ_RATIO: the paper's G = n / t (Problem Formulation), energy G * t_ref;
 *   a candidate is better iff n1 t2 > n2 t1.
 * level_len: proposals per temperature level; T is multiplied by alpha after each level
 *   (Algorithm 1 cools once per level of iter proposals), so T_k = T0 alpha^floor(k/L).
 * early_exit: Algorithm 1's first test -- when the solo-latency order meets every SLO it is
 *   the result; the chain makes no proposal. */
enum { ORC_OBJ_LEX = 0, ORC_OBJ_RATIO = 1 };
typedef struct {
  int32_t objective, level_len, early_exit, reserved;
} orc_search;

/* 1 iff key (n1, t1) is strictly better than (n2, t2) under the objective. */
int orc_better(const orc_search *s, int64_t n1, int64_t t1, int64_t n2, int64_t t2);

/* Metropolis for the ratio objective: num = n' t - n t' (exact int64); accept iff num >= 0
 * or u < exp(x), x = ((double)num * t_ref) / (((double)t * t') * T), u = w3 * 2^-32. */
int orc_accept_ratio(int64_t num, int64_t t_ref, int64_t t, int64_t t2, double T, uint32_t w3);

/* orc_accept (rule 0: a = delta, b = t_ref) or orc_accept_ratio (rule 1: a = num, b = t_ref,
 * c = t, d = t') for each of k elements; out[r] = 1 if accepted else 0. */
void orc_accept_many(int32_t rule, int64_t k, const int64_t *a, const int64_t *b, const int64_t *c,
                     const int64_t *d, const double *T, const uint32_t *w3, uint8_t *out);

/* Temperature levels of Algorithm 1: T = T0, then T *= tau after each level, until T <
 * T_thres (the first level always runs). Pinned: T0 500, T_thres 20, tau 0.95 -> 63. */
int32_t orc_levels(double T0, double T_thres, double tau);

/* orc_start / orc_anneal_chain / orc_anneal_chain_batches / orc_brute under search
 * settings (the plain functions use {ORC_OBJ_LEX, 1, 0}). With early_exit and a
 * solo-latency order that meets every SLO, the start is that order. */
int orc_start_ex(const orc_queue *q, const orc_model *m, const orc_search *s, uint16_t *start,
                 int64_t *t_ref, int64_t *start_n, int64_t *start_t);
void orc_anneal_chain_ex(const orc_queue *q, const orc_model *m, const orc_search *s,
                         const uint16_t *start, int64_t t_ref, int allmet, int32_t chain,
                         int32_t iters, double T0, double alpha, uint64_t seed, uint16_t *cur,
                         uint16_t *best, int64_t *rec, int64_t *trace);
int64_t orc_brute_ex(const orc_queue *q, const orc_model *m, const orc_search *s, int64_t *best_n,
                     int64_t *best_t, uint16_t *best_perm);

/* Solo latency of one request (its replay alone). */
int64_t orc_solo(const orc_queue *q, const orc_model *m, int32_t r);

/* ---- joint search over order and batch sizes (sized.c) ----
 * starts: one flag per position, 1 where a batch begins; starts[0] = 1 and every batch
 * holds at most max_batch requests. */

/* 1 iff starts is a valid batch layout of n positions with batches of at most B. */
int orc_check_starts(const uint8_t *starts, int32_t n, int32_t B);

/* Maximum-size layout: a batch starts at every multiple of B. */
void orc_max_starts(int32_t n, int32_t B, uint8_t *starts);

/* Step-by-step static timeline with the given batches (batch index from the cumulated
 * batch sizes, waiting time = earlier batch durations). Returns -1 and (-1, -1) when perm
 * is not a permutation or starts is not a valid layout. Pinned by hand-worked timelines
 * with unequal batch sizes, by orc_replay for maximum-size layouts, by the batch-size-1
 * closed form, and by within-batch order invariance. */
int orc_replay_batches(const orc_queue *q, const orc_model *m, const uint16_t *perm,
                       const uint8_t *starts, int64_t *n_met, int64_t *t_sum, int64_t *ttft,
                       int64_t *e2e);

/* Rows of k x n orders and k x n layouts; out is k x 2 (n_met, t_sum) or (-1, -1). */
void orc_eval_rows_batches(const orc_queue *q, const orc_model *m, const uint16_t *perms,
                           const uint8_t *starts, int64_t row0, int64_t rows, int64_t *out);

/* squeezeLastIter / delayNextIter at position i, in place. Return 1 if the move is
 * allowed and made, 0 (arrays untouched) otherwise. Pinned by worked examples and by
 * layout validity over random sequences of moves. */
int orc_squeeze(uint16_t *perm, uint8_t *starts, int32_t n, int32_t B, int32_t i);
int orc_delay(uint16_t *perm, uint8_t *starts, int32_t n, int32_t B, int32_t i);

/* Move choice of the joint search: floor(w0 * 3 / 2^32): 0 squeeze, 1 delay, 2 swap. */
int orc_op3(uint32_t w0);

/* One chain of the joint search: the start order of orc_start with maximum-size batches;
 * each iteration draws the Philox block of orc_anneal_chain, picks the move by orc_op3
 * (position i from w1 for squeeze and delay; i, j from w1, w2 for swap) and applies the
 * acceptance test of orc_accept. A move that is not allowed changes nothing and is not
 * counted as accepted. trace (nullable): iters x 4 int64 (accepted, n, t, move | 4 if not
 * allowed). Parity unpinned (trajectory). */
void orc_anneal_chain_batches(const orc_queue *q, const orc_model *m, const uint16_t *start,
                              int64_t t_ref, int allmet, int32_t chain, int32_t iters, double T0,
                              double alpha, uint64_t seed, uint16_t *cur, uint8_t *cur_starts,
                              uint16_t *best, uint8_t *best_starts, int64_t *rec, int64_t *trace);

/* Exhaustive search over every order and every layout (n <= 8): the optimum key, the
 * first optimal (order, layout) with orders in lexicographic order and, per order,
 * layouts by increasing bit mask of the starts at positions 1 .. n-1; returns the number
 * of optimal (order, layout) pairs. */
int64_t orc_brute_batches(const orc_queue *q, const orc_model *m, int64_t *best_n, int64_t *best_t,
                          uint16_t *best_perm, uint8_t *best_starts);

void orc_anneal_chain_batches_ex(const orc_queue *q, const orc_model *m, const orc_search *s,
                                 const uint16_t *start, int64_t t_ref, int allmet, int32_t chain,
                                 int32_t iters, double T0, double alpha, uint64_t seed,
                                 uint16_t *cur, uint8_t *cur_starts, uint16_t *best,
                                 uint8_t *best_starts, int64_t *rec, int64_t *trace);

/* ---- multiple instances (multi.c) ----
 * Instance assignment of the Scheduling Solution (1 <= instances <= 64): inst_out[r] for
 * every request in arrival order. capacity: tokens per instance. Pinned by hand-worked
 * assignments, round-robin for equal capacities, and per-iteration capacity bounds. */
void orc_assign(const orc_queue *q, int32_t instances, const int64_t *capacity, int32_t *inst_out);

/* ---- the fitted latency predictor taken literally (fit.c) ----
 * Per request in a static batch of b: t_p(b, l) = ap b l + bp b + cp l + dp; decode
 * sum_{k=1..L} tau_d(b, l + k), tau_d(b, l) = ad b l + bd b + cd l + dd; a batch lasts as
 * long as its slowest member. Kind ORC_TTFT_TPOT: TTFT <= thr and TPOT <= thr2 (the
 * paper's chat SLO), thr2 from a second array. All times in the caller's unit. */
enum { ORC_TTFT_TPOT = 3 };
typedef struct {
  int32_t max_batch, policy;  /* policy: ORC_STATIC (maximum-size batches) or ORC_STATIC_SEARCH */
  int64_t ap, bp, cp, dp, ad, bd, cd, dd;
  int64_t t_ref;              /* Metropolis scale; 0: total latency of the input order */
  uint64_t swap_threshold;    /* fixed-size batches: swap iff w0 < this, else insert */
} orc_fit_model;

int64_t orc_fit_prefill(const orc_fit_model *f, int64_t b, int64_t l);
int64_t orc_fit_decode(const orc_fit_model *f, int64_t b, int64_t l, int64_t L);

/* Timeline of one order (starts: nullable, maximum-size batches). (-1, -1) for an order
 * that is not a permutation, an invalid layout, a kind above 3, or kind 3 without thr2.
 * Pinned by hand-worked timelines with the paper's Table 2 coefficients, the closed form
 * of the decode sum, batch size 1 (Smith's rule) and the dual kind's two special cases. */
int orc_replay_fit(const orc_queue *q, const orc_fit_model *f, const uint16_t *perm, const uint8_t *starts,
                   const uint32_t *thr2, int64_t *n_met, int64_t *t_sum, int64_t *ttft, int64_t *e2e);

/* Start order (requests sorted by their latency alone, b = 1; the input order when it is
 * strictly better, unless the early exit applies) and one chain: fixed-size batches with
 * swap / insert moves, or searched batch sizes with squeeze / delay / swap, as the other
 * chains. Parity unpinned (trajectory). */
int orc_start_fit(const orc_queue *q, const orc_fit_model *f, const orc_search *s, const uint32_t *thr2,
                  uint16_t *start, int64_t *t_ref, int64_t *start_n, int64_t *start_t);
void orc_anneal_chain_fit(const orc_queue *q, const orc_fit_model *f, const orc_search *s, const uint32_t *thr2,
                          const uint16_t *start, int64_t t_ref, int allmet, int32_t chain, int32_t iters, double T0,
                          double alpha, uint64_t seed, uint16_t *cur, uint8_t *cur_starts, uint16_t *best,
                          uint8_t *best_starts, int64_t *rec);

#endif
