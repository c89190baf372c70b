/* sloanneal -- MI355X (gfx950) library for the data-parallel hot path of the SLO-aware
 * LLM request scheduler of Huang et al., "SLO-Aware Scheduling for Large Language Model
 * Inferences": simulated annealing over request priority orders (Algorithm 1), each
 * proposal scored by replaying a batched-serving timeline under the integer latency model.
 *
 * Conventions for every entry point:
 *   - array arguments are DEVICE pointers unless stated otherwise; the caller owns them
 *     (e.g. torch tensors) and the library never frees or retains them;
 *   - work is enqueued on the caller's stream and runs asynchronously; no call blocks,
 *     synchronises or reads device memory on the host, so calls may be enqueued behind
 *     other work on the stream;
 *   - every call checks its host arguments (sizes, pointers, model, settings) and returns
 *     SCHED_OK (0) or a negative SCHED_E* code, enqueueing nothing on an error. The
 *     contents of the device arrays (queue entries, instance indices, capacities) and the
 *     int64 range they imply are checked on the device by the call's first kernel, which
 *     also picks the integer widths and so the kernel that runs. A failure there makes the
 *     call's outputs read as its documentation says (rows (-2, code), best key (-2, code,
 *     -1), ...) with code SCHED_EINVAL or SCHED_ERANGE, and sched_status reports it;
 *   - the library keeps no global state: all annealing state lives in the caller's
 *     workspace, so calls on distinct workspaces and streams are independent;
 *   - latencies are int64 microseconds; results are bit-identical run to run.
 */
#ifndef SLOANNEAL_H
#define SLOANNEAL_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  SCHED_OK = 0,
  SCHED_EINVAL = -1, /* a size, pointer, parameter or queue entry is out of range */
  SCHED_ENOSPC = -2, /* workspace smaller than sched_ws_bytes(n, chains) */
  SCHED_ERANGE = -3, /* the queue and model could overflow the int64 clock or objective */
  SCHED_EHIP = -4    /* a HIP runtime call failed; sched_strerror gives its message */
};

/* SLO kinds (Problem Formulation, the SLO-met flag x_i): a request meets its SLO when
 * TTFT <= thr, or TPOT <= thr, or end-to-end latency <= thr. TPOT is the decode time
 * divided by the output length and is checked exactly as (e2e - TTFT) <= thr * l_out. */
enum { SCHED_TTFT = 0, SCHED_TPOT = 1, SCHED_E2E = 2 };

/* Admission policy. STATIC: consecutive groups of max_batch requests in priority order
 * form batches; a batch starts when the previous one has drained (batch index and
 * waiting time of the Problem Formulation). CONTINUOUS: a finished request frees its
 * slot, refilled from the priority order at the next iteration. STATIC_SEARCH: static
 * batches whose sizes (each 1 .. max_batch) are searched together with the order, the
 * argmax over positions and batch indices of the Problem Formulation, explored by the
 * squeeze and delay moves of Algorithm 1. Evaluated without a layout, and at the start
 * of every chain, its batches have the maximum size, which makes it STATIC. */
enum { SCHED_STATIC = 0, SCHED_CONTINUOUS = 1, SCHED_STATIC_SEARCH = 2 };

#define SCHED_MAX_N 1024
#define SCHED_MAX_BATCH 64
#define SCHED_THR_MAX 0xFFFFFFFEu /* largest accepted SLO threshold (us) */
#define SCHED_MAX_INSTANCES 64

/* Request queue, structure of arrays, n entries, DEVICE pointers (paper: newly arrived
 * jobs with input length, predicted output length, SLO kind and threshold). */
typedef struct {
  int32_t n;                /* 1 .. SCHED_MAX_N */
  const uint16_t *in_len;   /* input (prompt) tokens l_i */
  const uint16_t *out_len;  /* predicted output tokens l_o, >= 1 */
  const uint8_t *kind;      /* SCHED_TTFT / SCHED_TPOT / SCHED_E2E */
  const uint32_t *thr_us;   /* SLO threshold in microseconds (per token for TPOT), <= SCHED_THR_MAX */
} sched_queue_t;

/* Latency model in integer microseconds (Latency Predictor section, integer form) and
 * annealing constants. Host struct. All coefficients must be >= 0.
 *   prefill iteration of an admitted group = sum over the group of (p0 + p1 * l_in);
 *     decodes already running stall during it; the group's TTFT is its end;
 *   decode iteration = d0 + d1 * b + d2 * ctx, b = running requests, ctx = the sum of
 *     their context lengths; a request's k-th decode step has context l_in + k;
 *   a request ends with its l_out-th decode iteration. */
typedef struct {
  int32_t max_batch;        /* 1 .. SCHED_MAX_BATCH */
  int32_t policy;           /* SCHED_STATIC, SCHED_CONTINUOUS or SCHED_STATIC_SEARCH */
  int64_t p0, p1, d0, d1, d2;
  int64_t t_ref_us;         /* Metropolis latency scale; 0 => total latency of the input order */
  uint64_t swap_threshold;  /* proposal is a swap iff Philox word 0 < this (0 .. 2^32); 2^31 = 50/50;
                               unused by SCHED_STATIC_SEARCH, whose three moves are equally likely */
} sched_model_t;

/* Score K priority orders (objective of the Problem Formulation, kept as the integer
 * pair n = requests meeting their SLO, t = sum of end-to-end latencies).
 *   perms  : k x n uint16, row-major; row r is a priority order (position -> request id)
 *   out    : k x 2 int64 (n_met, t_sum); a row that is not a permutation of 0..n-1 gets
 *            (-1, -1)
 *   detail : nullable; k x n x 2 int64 (ttft, e2e) indexed by request id; rows that are
 *            not permutations are left untouched
 * Returns SCHED_EINVAL for k < 0, a null pointer, a bad queue descriptor or model.
 * Checked on the device: a queue entry out of range (l_out = 0, kind above SCHED_E2E,
 * threshold above SCHED_THR_MAX) makes every row read (-2, SCHED_EINVAL), a queue and model
 * that could overflow the int64 clock every row (-2, SCHED_ERANGE); detail is then left
 * untouched. k == 0 is a no-op (the queue is not read). */
int sched_eval(const sched_queue_t *queue, const sched_model_t *model, const uint16_t *perms,
               int64_t k, int64_t *out, int64_t *detail, hipStream_t stream);

/* Score K (order, batch layout) pairs under static admission with the given batches
 * (batch-size sequence b_0 .. b_{M-1} of the Problem Formulation: the batch index of a
 * position comes from the cumulated sizes, a batch waits for the previous one to drain).
 *   perms  : k x n uint16, row-major priority orders, as for sched_eval
 *   starts : k x n uint8, row-major; starts[r][p] = 1 where a batch begins at position p,
 *            else 0. A valid layout has starts[r][0] = 1 and every batch at most
 *            max_batch positions long
 *   out    : k x 2 int64 (n_met, t_sum); (-1, -1) if the order is not a permutation or the
 *            layout is not valid
 *   detail : nullable; k x n x 2 int64 (ttft, e2e) by request id; invalid rows untouched
 * model->policy must be SCHED_STATIC or SCHED_STATIC_SEARCH (SCHED_EINVAL otherwise);
 * other errors, and the device checks of the queue, as for sched_eval. */
int sched_eval_batches(const sched_queue_t *queue, const sched_model_t *model, const uint16_t *perms,
                       const uint8_t *starts, int64_t k, int64_t *out, int64_t *detail, hipStream_t stream);

/* Bytes of workspace sched_anneal needs for n requests and `chains` chains (0 on bad sizes). */
size_t sched_ws_bytes(int32_t n, int32_t chains);

/* Run `chains` independent annealing chains of `iters` proposals each (Algorithm 1 with a
 * geometric schedule T_k = T0 * alpha^k, one proposal per iteration). All chains start
 * from the Algorithm 1 start order: requests sorted by solo latency (stable), replaced by
 * the input order when that scores strictly better. Proposal k of chain c uses the
 * Philox4x32-10 block with counter (k, c, 0, 0x53414E4E) and key (seed low, seed high):
 * word 0 picks swap or insert, words 1 and 2 the positions, word 3 the acceptance draw.
 * A worse candidate is accepted iff w3 * 2^-32 < exp(delta / (t_ref * T_k)) with
 * delta = (n' - n) * t_ref - (t' - t); others are always accepted. Each chain tracks its
 * best-so-far order (attainment first, then lower total latency); the best over chains
 * (lowest chain id on ties) is reduced at the end.
 *   ws : DEVICE workspace of at least sched_ws_bytes(n, chains) bytes, 256-byte aligned;
 *        it holds the start order, per-chain records and orders after the call.
 * With model->policy == SCHED_STATIC_SEARCH the state is the order and its batch layout
 * (Algorithm 1's joint search): every chain starts from the start order with maximum-size
 * batches, and proposal k picks move floor(w0 * 3 / 2^32): 0 squeezeLastIter (the request
 * at position i = floor(w1 * n / 2^32) joins the batch before its own as its last member,
 * allowed when its batch is not the first and the one before holds fewer than max_batch),
 * 1 delayNextIter (it joins the batch after its own as its first member, allowed when that
 * batch holds fewer than max_batch; from the last batch it opens a new one, allowed when
 * it does not run alone), 2 a swap of positions i and j (as above). A move that is not
 * allowed changes nothing and counts as neither accepted nor rejected (no digest step).
 * Layouts are read back with sched_starts.
 * Returns SCHED_EINVAL for chains < 1, iters < 0, T0 <= 0, alpha <= 0 or non-finite,
 * a bad queue descriptor or model; SCHED_ENOSPC for a short workspace. Checked on the
 * device: a queue entry out of range (SCHED_EINVAL) or overflow risk of the int64 clock
 * (SCHED_ERANGE) ends the call after its first kernel; sched_status then reads the code,
 * sched_best's key (-2, code, -1), sched_chains' records (-2, code, -1, ...) and
 * sched_start_info's info (-2, code, -1, -1), and the orders in ws are not written. */
int sched_anneal(const sched_queue_t *queue, const sched_model_t *model, int32_t chains,
                 int32_t iters, double T0, double alpha, uint64_t seed, void *ws, size_t ws_bytes,
                 hipStream_t stream);

/* Search settings of Algorithm 1 beyond the workloads' defaults.
 *   objective  : SCHED_OBJ_LEX (default): attainment first, then lower total latency, with
 *                Metropolis energy n - t / t_ref. SCHED_OBJ_RATIO: the paper's objective
 *                G = n / t (Problem Formulation), energy G * t_ref; a worse candidate is kept
 *                iff w3 * 2^-32 < exp(x), x = (num * t_ref) / ((t * t') * T_k) in double
 *                arithmetic in that order, num = n' t - n t'; keys compare by n1 t2 vs n2 t1
 *                (best-so-far, the cross-chain winner and the start rule alike). Needs
 *                p0 + d0 + d1 >= 1 (a positive total latency).
 *   level_len  : proposals per temperature level, >= 1: T_k = T0 * alpha^floor(k / level_len)
 *                (Algorithm 1 lowers T once per level of `iter` proposals; 1 = per proposal).
 *   early_exit : 1 = Algorithm 1's first test: when the requests sorted by solo latency meet
 *                every SLO, that order is the start and the result and no proposal runs.
 *   reserved   : 0. */
enum { SCHED_OBJ_LEX = 0, SCHED_OBJ_RATIO = 1 };
typedef struct {
  int32_t objective, level_len, early_exit, reserved;
} sched_search_t;

/* sched_anneal with search settings (search == NULL: {SCHED_OBJ_LEX, 1, 0, 0}, which is
 * sched_anneal). The paper's schedule (T0 500, T_thres 20, tau 0.95, iter 100) is
 * T0 = 500, alpha = 0.95, level_len = 100, iters = 100 * sched_levels(500, 20, 0.95).
 * Errors as sched_anneal, and SCHED_EINVAL for bad settings; on the device SCHED_ERANGE
 * also when the ratio's int64 cross products could overflow. */
int sched_anneal_ex(const sched_queue_t *queue, const sched_model_t *model, const sched_search_t *search,
                    int32_t chains, int32_t iters, double T0, double alpha, uint64_t seed, void *ws,
                    size_t ws_bytes, hipStream_t stream);

/* Number of temperature levels of Algorithm 1: T starts at T0 and is multiplied by tau after
 * each level until it falls below T_thres (the first level always runs); computed on the
 * host by repeated double multiplication. SCHED_EINVAL for T0 or T_thres not positive and
 * finite, or tau outside (0, 1). */
int32_t sched_levels(double T0, double T_thres, double tau);

/* ---- the Latency Predictor's fitted model taken literally ----
 * Each member of a static batch of b requests has its own prediction (equations for t_p,
 * tau_d and t_d, with their batch-size interaction terms): prefill
 *   t_p(b, l) = ap * b * l + bp * b + cp * l + dp,
 * decode summed over its l_out tokens of tau_d(b, l + k) = ad * b * (l + k) + bd * b +
 * cd * (l + k) + dd; TTFT = wait + t_p, e2e = wait + t_p + t_d, TPOT = t_d / l_out. A batch
 * lasts as long as its slowest member and waits for every earlier batch. Coefficients are
 * integers >= 0 in one time unit of the caller's choice, thresholds in the same unit (the
 * paper's Table 2, in ms, is exact in units of 10 ns: ap 10000, bp 570000, cp 1000,
 * dp 4367000, ad 20, bd 27500, cd 88, dd 1585000). Host struct. */
typedef struct {
  int32_t max_batch;        /* 1 .. SCHED_MAX_BATCH */
  int32_t policy;           /* SCHED_STATIC (maximum-size batches) or SCHED_STATIC_SEARCH */
  int64_t ap, bp, cp, dp;   /* prefill */
  int64_t ad, bd, cd, dd;   /* per-token decode */
  int64_t t_ref;            /* Metropolis latency scale; 0 => total latency of the input order */
  uint64_t swap_threshold;  /* SCHED_STATIC: swap iff Philox word 0 < this, else insert */
} sched_fit_model_t;

/* The paper's chat SLO (the definition of x_i for h_i = 0): TTFT <= thr_us AND
 * TPOT <= tpot_thr, the second threshold from the tpot_thr array of the fitted-model calls. */
enum { SCHED_TTFT_TPOT = 3 };

/* sched_eval / sched_eval_batches under the fitted model.
 *   tpot_thr : nullable DEVICE n x uint32, the TPOT thresholds of SCHED_TTFT_TPOT requests
 *              (a queue with that kind fails the device check, SCHED_EINVAL, when it is null)
 *   starts   : nullable DEVICE k x n uint8 batch layouts (as for sched_eval_batches); null =
 *              maximum-size batches
 * Other arguments, outputs and errors as for sched_eval_batches (the device check of the
 * kinds accepts SCHED_TTFT_TPOT when tpot_thr is given; SCHED_ERANGE when the latencies
 * could overflow int64). */
int sched_eval_fit(const sched_queue_t *queue, const sched_fit_model_t *fit, const uint32_t *tpot_thr,
                   const uint16_t *perms, const uint8_t *starts, int64_t k, int64_t *out, int64_t *detail,
                   hipStream_t stream);

/* sched_anneal_ex under the fitted model: the start order sorts requests by their latency
 * alone (b = 1); fixed-size batches take swap / insert proposals and SCHED_STATIC_SEARCH the
 * squeeze / delay / swap moves (layouts read back with sched_starts); every proposal is
 * replayed in full. Readouts as for sched_anneal. The ratio objective needs dp + dd >= 1. */
int sched_anneal_fit(const sched_queue_t *queue, const sched_fit_model_t *fit, const uint32_t *tpot_thr,
                     const sched_search_t *search, int32_t chains, int32_t iters, double T0, double alpha,
                     uint64_t seed, void *ws, size_t ws_bytes, hipStream_t stream);

/* ---- several serving instances (Scheduling Solution section, Algorithm 2) ----
 * Callers: a scheduler in front of several LLM instances that first assigns the newly
 * arrived requests to instances and then orders each instance's requests. */

/* Instance assignment (InstAssign): requests in arrival order, each to the instance with
 * the largest remaining memory in tokens; a request holds in_len + out_len tokens. When
 * even that instance cannot hold the request, every instance's remaining memory is reset
 * to its capacity (a fresh iteration) and the request goes to the instance with the largest
 * capacity, even if it does not fit there. Ties go to the lowest index.
 *   capacity : DEVICE, instances x int64 tokens per instance (token_num(m) = m * mu / sigma,
 *              computed by the caller), each 1 .. 2^48
 *   inst_out : DEVICE, n x int32, the instance of every request
 * SCHED_EINVAL for instances outside 1 .. SCHED_MAX_INSTANCES, null pointers or a bad queue
 * descriptor. Checked on the device: a queue entry or a capacity out of range makes every
 * entry of inst_out read SCHED_EINVAL. */
int sched_assign(const sched_queue_t *queue, int32_t instances, const int64_t *capacity, int32_t *inst_out,
                 hipStream_t stream);

/* Bytes of workspace sched_anneal_multi needs (0 on bad sizes). */
size_t sched_ws_bytes_multi(int32_t n, int32_t instances, int32_t chains);

/* Priority mapping within every instance independently, all instances side by side: the
 * requests with inst_of[r] == k, in arrival order, form instance k's queue, and instance k
 * runs `chains` chains on it exactly as sched_anneal_ex would on that queue, except that
 * its chain c draws from Philox chain index k * chains + c. One launch per step covers every
 * instance (chains by full replay of each proposal). model->policy must be SCHED_STATIC or
 * SCHED_CONTINUOUS; search as for sched_anneal_ex (NULL for the defaults).
 *   inst_of : DEVICE, n x int32 in 0 .. instances - 1 (e.g. from sched_assign)
 *   ws      : DEVICE, at least sched_ws_bytes_multi(n, instances, chains) bytes, 256-aligned
 * Instance k's chains are read with sched_best / sched_chains / sched_start_info on
 * sched_multi_instance_ws(ws, ...k); their orders index the instance's own queue. An
 * instance with no request runs nothing. Errors as sched_anneal_ex; the device checks also
 * reject an inst_of entry outside 0 .. instances - 1 (SCHED_EINVAL), and after a failed
 * check sched_status(ws) reads the code, sched_multi_best's keys (-2, code, -1) with counts
 * 0 and orders untouched, and each instance workspace reads as a failed sched_anneal's. */
int sched_anneal_multi(const sched_queue_t *queue, const sched_model_t *model, const sched_search_t *search,
                       const int32_t *inst_of, int32_t instances, int32_t chains, int32_t iters, double T0,
                       double alpha, uint64_t seed, void *ws, size_t ws_bytes, hipStream_t stream);

/* Instance k's single-queue workspace inside a sched_anneal_multi workspace (pointer
 * arithmetic only; NULL on bad arguments). */
void *sched_multi_instance_ws(void *ws, int32_t n, int32_t instances, int32_t chains, int32_t instance);

/* Every instance's best order, as global request ids, instance after instance.
 *   orders : DEVICE, n x uint16: instance 0's requests in its best priority order, then
 *            instance 1's, ...
 *   keys   : DEVICE nullable, instances x 3 int64 (n_met, t_sum, chain); (-1, -1, -1) for an
 *            instance without requests
 *   counts : DEVICE nullable, instances x int32 requests per instance
 * (Scheduling Solution section: the per-instance results of Algorithm 2's priority
 * mapping.) */
int sched_multi_best(const void *ws, int32_t instances, uint16_t *orders, int64_t *keys, int32_t *counts,
                     hipStream_t stream);

/* ---- no device allocation ----
 * For callers that cannot allocate device memory (code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc): sched_anneal followed by sched_best, with
 * the annealing workspace in a fixed scratch array that the library holds on every GPU it
 * runs on (SCHED_NOALLOC_MAX_BYTES per GPU, kept until the process ends) instead of a
 * caller's workspace. The call allocates nothing. Every call on one GPU shares that GPU's
 * scratch and leaves its contents there (nothing in it has to start at zero: each call
 * writes what it later reads), so calls that overlap on one GPU race: serialise them, e.g.
 * on one stream. The stream must belong to the current device.
 *   perm_out : n uint16 (DEVICE), the best order over chains; key_out : 3 int64 (DEVICE) =
 *              (n_met, t_sum, chain), as sched_best returns them.
 * Arguments otherwise and errors as sched_anneal; SCHED_ENOSPC when sched_ws_bytes(n,
 * chains) exceeds SCHED_NOALLOC_MAX_BYTES (it holds up to 5404 chains of 1024 requests,
 * 20971 of 256 and 30840 of 128 or fewer). */
#define SCHED_NOALLOC_MAX_BYTES (32u << 20)
int sched_anneal_noalloc(const sched_queue_t *queue, const sched_model_t *model, int32_t chains, int32_t iters,
                         double T0, double alpha, uint64_t seed, uint16_t *perm_out, int64_t *key_out,
                         hipStream_t stream);

/* Best order over all chains of the last sched_anneal on ws: the priority order Algorithm 1
 * returns (Priority Mapping Algorithm section), taken as the best of every chain's
 * best-so-far order (attainment first, then lower total latency; lowest chain id on ties).
 *   perm_out : n uint16 (DEVICE); key_out : 3 int64 (DEVICE) = (n_met, t_sum, chain); after
 *   a call whose device checks failed the key reads (-2, code, -1) and perm_out is left
 *   untouched. */
int sched_best(const void *ws, uint16_t *perm_out, int64_t *key_out, hipStream_t stream);

/* Per-chain readout of the last sched_anneal on ws (observability and parity checks).
 *   per_chain  : chains x 8 int64 (DEVICE) = (cur n, cur t, best n, best t, best iteration
 *                or -1, accepted proposals, trajectory digest, start-order-meets-all flag)
 *   cur_perms  : nullable, chains x n uint16 final orders
 *   best_perms : nullable, chains x n uint16 best orders
 * The digest folds (iteration, n, t) of every accepted proposal, in order, with 64-bit
 * FNV-1a steps: d = (d ^ word) * 0x100000001B3, starting at 0xCBF29CE484222325. */
int sched_chains(const void *ws, int64_t *per_chain, uint16_t *cur_perms, uint16_t *best_perms,
                 hipStream_t stream);

/* Start order and constants of the last sched_anneal on ws.
 *   start_out : n uint16 (DEVICE); info_out : 4 int64 (DEVICE) = (t_ref, start n, start t,
 *               1 if the solo-latency order meets every SLO else 0). */
int sched_start_info(const void *ws, uint16_t *start_out, int64_t *info_out, hipStream_t stream);

/* Batch layouts of the last sched_anneal on ws with SCHED_STATIC_SEARCH (start flags,
 * one uint8 per position as for sched_eval_batches). After a run with another policy every
 * layout reads as the maximum-size one (a start at every multiple of max_batch). All
 * outputs DEVICE and nullable, at least one given (SCHED_EINVAL otherwise):
 *   cur_starts    : chains x n, each chain's final layout
 *   best_starts   : chains x n, each chain's best-so-far layout
 *   winner_starts : n, the layout of the best order over chains (the one sched_best returns) */
int sched_starts(const void *ws, uint8_t *cur_starts, uint8_t *best_starts, uint8_t *winner_starts,
                 hipStream_t stream);

/* Fill rows row0 .. row0+k-1 of a Fisher-Yates permutation family: row r shuffles 0..n-1
 * for positions p = n-1 down to 1 with j = (w * (p + 1)) >> 32, w = word (p mod 4) of the
 * Philox4x32-10 block with counter (p / 4, r, 1, 0x46495348) and key (seed low, seed high).
 *   perms : k x n uint16 (DEVICE), row-major. */
int sched_gen_perms(uint64_t seed, int32_t n, int64_t row0, int64_t k, uint16_t *perms,
                    hipStream_t stream);

/* The acceptance step of Algorithm 1 (Priority Mapping Algorithm section) as the annealing
 * kernels evaluate it, on caller-given inputs: a test and observability readout, so that
 * the single-precision screen in front of the double-precision rule can be compared with a
 * reference decision by decision. All arrays DEVICE, k elements:
 *   rule 0 : a = delta, b = t_ref (>= 1); keep iff delta >= 0 or
 *            w3 * 2^-32 < exp(delta / (t_ref * T)) (the rule of sched_anneal);
 *   rule 1 : a = num, b = t_ref, c = t, d = t' (t, t' >= 1); keep iff num >= 0 or
 *            w3 * 2^-32 < exp((num * t_ref) / ((t * t') * T)) (SCHED_OBJ_RATIO);
 *   c, d   : used by rule 1 only (nullable for rule 0); T > 0;
 *   out    : bit 0 = kept; bit 1 = decided by the single-precision screen (else the
 *            double-precision rule decided, or the candidate was not worse).
 * SCHED_EINVAL for another rule, k < 0 or a null array that the rule reads. */
int sched_accept_check(int32_t rule, int64_t k, const int64_t *a, const int64_t *b, const uint64_t *c,
                       const uint64_t *d, const double *T, const uint32_t *w3, uint8_t *out, hipStream_t stream);

/* The device checks' verdict of the last annealing call on ws (a sched_anneal* workspace, a
 * sched_anneal_multi workspace or an instance workspace inside one): an observability
 * readout for the asynchronous calls.
 *   out : 3 int64 (DEVICE) = (status: SCHED_OK, SCHED_EINVAL or SCHED_ERANGE; the integer
 *         widths that hold for the queue, a bit set; the index of the kernel that ran among
 *         the call's candidates, -1 when the checks failed). */
int sched_status(const void *ws, int64_t *out, hipStream_t stream);

/* Static message for a SCHED_* code; for SCHED_EHIP the last HIP error seen by this thread. */
const char *sched_strerror(int code);

#ifdef __cplusplus
}
#endif
#endif
