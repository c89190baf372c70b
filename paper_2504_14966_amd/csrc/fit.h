// The Latency Predictor's fitted model taken literally (gfx950, wave64).
//
// Each member of a static batch of b requests has its own prediction: prefill
//   t_p(b, l) = ap b l + bp b + cp l + dp,
// and decode summed over its L output tokens of tau_d(b, l + k) = ad b (l + k) + bd b +
// cd (l + k) + dd, which is in closed form
//   t_d = L (bd b + dd) + (ad b + cd) (L l + L (L + 1) / 2).
// TTFT = wait + t_p, e2e = wait + t_p + t_d, TPOT = t_d / L; a batch lasts as long as its
// slowest member and waits for every earlier batch. Coefficients are integers in the
// caller's time unit (the paper's Table 2, in milliseconds, is exact in units of 10 ns).
//
// SLO kinds: the three single ones and kind 3, the paper's chat SLO (TTFT <= thr and TPOT
// <= thr2, thr2 from a second per-request array).
//
// Batches are either of the maximum size or given by start flags (the batch-size search),
// and every proposal is replayed in full, one batch at a time with the members in lanes:
// per member one closed form, per batch a wave maximum. All arithmetic is 64-bit.
#pragma once
#include "anneal_sized.h"

namespace sa {

struct DevFit {
  int32_t n, B, policy, pad;
  uint64_t ap, bp, cp, dp, ad, bd, cd, dd;
  uint32_t win;  // 1: every member's time is below 2^57 (the windowed replay's keys fit)
  uint32_t m32;  // 1: every member's time, in any batch, is below 2^32 - 1
  uint64_t bmagic;     // floor(2^32 / B) + 1: lane / B = (lane * bmagic) >> 32 for lanes below 64
  // for the device checks of the queue, which set win and m32 where the gate allows them
  int64_t t_ref;     // the caller's Metropolis scale (0: total latency of the input order)
  int32_t max_kind;  // largest SLO kind accepted (3 with the second threshold array)
  int32_t ratio;     // 1: the ratio objective
  Gate gate;
};

// The device checks under the fitted model, formed by the whole workgroup.
__device__ __forceinline__ Plan fit_plan_in_block(const QueuePtrs &q, const DevFit &f) {
  const FitCoef c{f.ap, f.bp, f.cp, f.dp, f.ad, f.bd, f.cd, f.dd};
  const QueueStats s = block_queue_stats(q, f.n, f.B, f.max_kind, &c);
  Plan p = plan_decide(s, f.n, f.B, f.ratio, f.t_ref, 0, 0, 0, 0, 0, &c, f.gate);
  if (p.status == 0) p.selected = plan_select(f.gate, p.flags);
  return p;
}
__device__ __forceinline__ void fit_take_flags(DevFit &f, uint32_t flags) {
  const uint32_t a = flags & f.gate.allow;
  f.win = (a & kFlagFitWindows) ? 1u : 0u;
  f.m32 = (a & kFlagFitMember32) ? 1u : 0u;
}
// As gate_open, for the fitted-model kernels.
__device__ __forceinline__ bool fit_gate_open(const unsigned char *ws, DevFit &f) {
  const WsHeader *h = reinterpret_cast<const WsHeader *>(ws);
  if (h->plan_selected != (int64_t)f.gate.self) return false;
  fit_take_flags(f, (uint32_t)h->plan_flags);
  return true;
}
// As eval_gate, for the fitted-model evaluation.
__device__ __forceinline__ EvalRows eval_fit_gate(const QueuePtrs &q, DevFit &f, int64_t rows, int64_t *out) {
  uint32_t flags = 0u;
  const EvalRows r = eval_rows_of([&]() { return fit_plan_in_block(q, f); }, f.gate, rows, out, flags);
  fit_take_flags(f, flags);
  return r;
}

// Request record: x = l_in | l_out << 16, y = threshold, z = kind, w = second threshold.
__device__ __forceinline__ void load_fit_requests(const QueuePtrs &q, const uint32_t *thr2, int n, uint4 *req) {
  for (int r = threadIdx.x; r < n; r += blockDim.x) {
    const uint32_t lin = q.in_len[r], lout = q.out_len[r];
    req[r] = make_uint4(lin | (lout << 16), q.thr[r], (uint32_t)q.kind[r], thr2 ? thr2[r] : 0u);
  }
}

__device__ __forceinline__ uint64_t fit_prefill(const DevFit &f, uint64_t b, uint64_t l) {
  return f.ap * b * l + f.bp * b + f.cp * l + f.dp;
}
__device__ __forceinline__ uint64_t fit_decode(const DevFit &f, uint64_t b, uint64_t l, uint64_t L) {
  return L * (f.bd * b + f.dd) + (f.ad * b + f.cd) * (L * l + L * (L + 1) / 2);
}

__device__ __forceinline__ bool fit_met(uint32_t kind, uint64_t thr, uint64_t thr2, uint64_t L, uint64_t ttft,
                                        uint64_t td, uint64_t e2e) {
  if (kind == 0) return ttft <= thr;
  if (kind == 2) return e2e <= thr;
  if (kind == 1) return td <= thr * L;
  return ttft <= thr && td <= thr2 * L;
}

// flags: start flags of the layout, or null for batches of the maximum size. One batch at
// a time (any member time).
template <bool DETAIL>
__device__ Score replay_fit_batches(const DevFit &f, const uint4 *__restrict__ req, const uint16_t *perm,
                                    const uint8_t *flags, int64_t *detail) {
  const int lane = lane_id();
  const int n = f.n;
  uint64_t S = 0, tl = 0;
  int64_t nmet = 0;
  for (int s = 0; s < n;) {
    const int e = flags ? batch_end(flags, n, s, lane) : min(n, s + f.B);
    const int b = e - s;
    const bool valid = lane < b;
    uint64_t exec = 0;
    bool met = false;
    if (valid) {
      const int r = perm[s + lane];
      const uint4 rq = req[r];
      const uint64_t l = rq.x & 0xFFFFu, L = rq.x >> 16;
      const uint64_t tp = fit_prefill(f, (uint64_t)b, l), td = fit_decode(f, (uint64_t)b, l, L);
      exec = tp + td;
      const uint64_t ttft = S + tp, e2e = S + exec;
      met = fit_met(rq.z, rq.y, rq.w, L, ttft, td, e2e);
      tl += e2e;
      if (DETAIL) {
        detail[2 * r] = (int64_t)ttft;
        detail[2 * r + 1] = (int64_t)e2e;
      }
    }
    nmet += ballot_count(met);
    S += wave_max_u64(exec);
    s = e;
  }
  return Score{nmet, wave_sum_u64(tl)};
}

// The same timeline over windows of whole batches: a window starts at a batch start and
// takes every batch that ends within the next 64 positions, one position per lane. A lane's
// batch and size come from the mask of batch-last lanes; its time from the closed forms.
// The batch durations are one max-scan of the key (batch start lane << 58 | time): batch
// starts never decrease across lanes, so the running maximum of the key at a lane is the
// running maximum of the time within the lane's own batch, and at the batch's last lane its
// duration (needs every time below 2^58). The batches' start times are one add-scan of the
// durations at the batch-last lanes.
template <bool DETAIL>
__device__ Score replay_fit_windows(const DevFit &f, const uint4 *__restrict__ req, const uint16_t *perm,
                                    const uint8_t *flags, int64_t *detail) {
  const int lane = lane_id();
  const int n = f.n, B = f.B;
  constexpr uint64_t kTimeMask = (uint64_t(1) << 58) - 1;
  uint64_t S0 = 0, tl = 0;
  int64_t nmet = 0;
  for (int s = 0; s < n;) {
    const int p = s + lane;
    // lane begins a batch (lane 0 always does) or is the end of the queue
    bool st = p == n;
    if (p < n) {
      if (flags) st = lane == 0 || flags[p] != 0;
      else st = (uint64_t)lane == (((uint64_t)lane * f.bmagic) >> 32) * (uint64_t)B;
    }
    // position s + 64 begins a batch or is the end of the queue
    bool st64 = s + kWave == n;
    if (s + kWave < n) st64 = flags ? flags[s + kWave] != 0 : (kWave % B) == 0;
    uint64_t lastm = (__ballot(st) >> 1) | (st64 ? uint64_t(1) << 63 : 0ull);  // batch-last lanes
    // a valid layout always closes a batch within 64 positions; a malformed one is cut
    // there so that the window advances
    if (lastm == 0ull) lastm = uint64_t(1) << 63;
    const int w = 64 - __clzll(lastm);  // lanes [0, w) hold whole batches
    const bool in = lane < w;
    const uint64_t below = lastm & ((uint64_t(1) << lane) - 1);
    const int b0 = below ? 64 - __clzll(below) : 0;              // first lane of the lane's batch
    const int b1 = lane + __builtin_ctzll(in ? (lastm >> lane) : 1ull);  // its last lane
    uint64_t tp = 0, E = 0;
    uint4 rq = make_uint4(0u, 0u, 0u, 0u);
    int r = 0;
    if (in) {
      r = perm[p];
      rq = req[r];
      const uint64_t b = (uint64_t)(b1 - b0 + 1), l = rq.x & 0xFFFFu, L = rq.x >> 16;
      tp = fit_prefill(f, b, l);
      E = tp + fit_decode(f, b, l, L);
    }
    const uint64_t D = scan_max64(in ? ((uint64_t)b0 << 58) | E : 0ull) & kTimeMask;
    const uint64_t contrib = (in && lane == b1) ? D : 0ull;
    const uint64_t incl = scan_add64(contrib);
    const uint64_t S = S0 + (incl - contrib);
    bool met = false;
    if (in) {
      const uint64_t L = rq.x >> 16, ttft = S + tp, e2e = S + E;
      met = fit_met(rq.z, rq.y, rq.w, L, ttft, E - tp, e2e);
      tl += e2e;
      if (DETAIL) {
        detail[2 * r] = (int64_t)ttft;
        detail[2 * r + 1] = (int64_t)e2e;
      }
    }
    nmet += ballot_count(met);
    S0 += rl64(incl, kWave - 1);
    s += w;
  }
  return Score{nmet, wave_sum_u64(tl)};
}

// The same windows when every member's time fits 32 bits (totals only): the closed forms in
// 32-bit arithmetic (exact, the wrap-around only inside ring expressions whose value fits),
// durations by the 32-bit max-scan confined to batches, starts by saturating 32-bit scans
// (a start that saturates meets no threshold, every threshold being below 2^32 - 1), and
// the total latency exactly as the sum of the member times plus each batch's duration times
// the number of requests after it.
__device__ Score replay_fit_windows32(const DevFit &f, const uint4 *__restrict__ req, const uint16_t *perm,
                                      const uint8_t *flags) {
  const int lane = lane_id();
  const int n = f.n, B = f.B;
  const uint32_t ap = (uint32_t)f.ap, bp = (uint32_t)f.bp, cp = (uint32_t)f.cp, dp = (uint32_t)f.dp;
  const uint32_t ad = (uint32_t)f.ad, bd = (uint32_t)f.bd, cd = (uint32_t)f.cd, dd = (uint32_t)f.dd;
  uint32_t S0 = 0;    // start of the window, saturated
  uint64_t tsum = 0;  // per lane: member times and duration-weighted counts
  int64_t nmet = 0;
  for (int s = 0; s < n;) {
    const int p = s + lane;
    bool st = p == n;
    if (p < n) {
      if (flags) st = lane == 0 || flags[p] != 0;
      else st = (uint64_t)lane == (((uint64_t)lane * f.bmagic) >> 32) * (uint64_t)B;
    }
    bool st64 = s + kWave == n;
    if (s + kWave < n) st64 = flags ? flags[s + kWave] != 0 : (kWave % B) == 0;
    uint64_t lastm = (__ballot(st) >> 1) | (st64 ? uint64_t(1) << 63 : 0ull);
    if (lastm == 0ull) lastm = uint64_t(1) << 63;
    const int w = 64 - __clzll(lastm);
    const bool in = lane < w;
    const uint64_t below = lastm & ((uint64_t(1) << lane) - 1);
    const int b0 = below ? 64 - __clzll(below) : 0;
    const int b1 = lane + __builtin_ctzll(in ? (lastm >> lane) : 1ull);
    uint32_t tp = 0, td = 0, E = 0, L = 0;
    uint4 rq = make_uint4(0u, 0u, 0u, 0u);
    if (in) {
      rq = req[perm[p]];
      const uint32_t b = (uint32_t)(b1 - b0 + 1), l = rq.x & 0xFFFFu;
      L = rq.x >> 16;
      tp = ap * b * l + bp * b + cp * l + dp;
      td = L * (bd * b + dd) + (ad * b + cd) * (L * l + ((L * (L + 1u)) >> 1));
      E = tp + td;
    }
    // lanes past the window hold E = 0 and send nothing; what they receive is unused
    const uint32_t D = seg_max32(E, b0, b1, lane);
    const bool last = in && lane == b1;
    const uint32_t contrib = last ? D : 0u;
    // durations of the window's earlier batches: the inclusive scan moved up one lane
    const uint32_t excl =
        scan_add_sat32((uint32_t)__builtin_amdgcn_update_dpp(0, (int)contrib, kDppWaveShr1, 0xF, 0xF, false));
    const uint32_t S = add_sat(S0, excl);
    bool met = false;
    if (in) {
      const uint32_t ttft = add_sat(S, tp), e2e = add_sat(S, E);
      const uint32_t kind = rq.z;
      met = kind == 0   ? ttft <= rq.y
            : kind == 1 ? (uint64_t)td <= (uint64_t)rq.y * L
            : kind == 2 ? e2e <= rq.y
                        : (ttft <= rq.y && (uint64_t)td <= (uint64_t)rq.w * L);
    }
    nmet += ballot_count(met);
    tsum += (uint64_t)E + (uint64_t)contrib * (uint32_t)(last ? n - 1 - p : 0);
    S0 = add_sat(S0, add_sat(readlane(excl, kWave - 1), readlane(contrib, kWave - 1)));
    s += w;
  }
  return Score{nmet, wave_sum_u64(tsum)};
}

template <bool DETAIL>
__device__ __forceinline__ Score replay_fit(const DevFit &f, const uint4 *__restrict__ req, const uint16_t *perm,
                                            const uint8_t *flags, int64_t *detail) {
  if constexpr (!DETAIL) {
    if (f.m32) return replay_fit_windows32(f, req, perm, flags);
  }
  if (f.win) return replay_fit_windows<DETAIL>(f, req, perm, flags, detail);
  return replay_fit_batches<DETAIL>(f, req, perm, flags, detail);
}

// K rows: one wave per row; rows validated first ((-1, -1) otherwise). starts nullable.
template <bool DETAIL>
__global__ void __launch_bounds__(256) eval_fit_kernel(DevFit f, QueuePtrs q, const uint32_t *__restrict__ thr2,
                                                        const uint16_t *__restrict__ perms,
                                                        const uint8_t *__restrict__ starts, int64_t rows,
                                                        int64_t *__restrict__ out, int64_t *__restrict__ detail) {
  extern __shared__ __align__(16) unsigned char lds[];
  const EvalRows span = eval_fit_gate(q, f, rows, out);
  if (span.end <= span.begin) return;
  const int n = f.n;
  uint4 *req = reinterpret_cast<uint4 *>(lds);
  const size_t pb = ((size_t)n * 2 + 15) & ~size_t(15), fb = ((size_t)n + 15) & ~size_t(15);
  const size_t per_wave = pb + fb + 32 * 4;
  const int wave = uniform((int)(threadIdx.x >> 6));
  unsigned char *wb = lds + (((size_t)n * 16 + 15) & ~size_t(15)) + (size_t)wave * per_wave;
  uint16_t *perm = reinterpret_cast<uint16_t *>(wb);
  uint8_t *flags = wb + pb;
  uint32_t *bitmap = reinterpret_cast<uint32_t *>(wb + pb + fb);
  load_fit_requests(q, thr2, n, req);
  __syncthreads();
  const int lane = lane_id();
  const int waves = blockDim.x >> 6;
  for (int64_t row = span.begin + (int64_t)blockIdx.x * waves + wave; row < span.end;
       row += (int64_t)gridDim.x * waves) {
    const uint16_t *src = perms + row * n;
    if (lane < 32) bitmap[lane] = 0u;
    wave_sync_lds();
    bool bad = false;
    for (int p = lane; p < n; p += kWave) {
      const uint32_t v = src[p];
      perm[p] = (uint16_t)v;
      if (starts) flags[p] = starts[row * n + p];
      if (v >= (uint32_t)n) {
        bad = true;
      } else {
        const uint32_t bit = 1u << (v & 31u);
        const uint32_t old = atomicOr(&bitmap[v >> 5], bit);
        if (old & bit) bad = true;
      }
    }
    wave_sync_lds();
    const bool ok = __ballot(bad) == 0ull && (!starts || layout_ok(flags, n, f.B, lane));
    if (!ok) {
      if (lane == 0) {
        out[2 * row] = -1;
        out[2 * row + 1] = -1;
      }
      continue;
    }
    const Score s =
        replay_fit<DETAIL>(f, req, perm, starts ? flags : nullptr, DETAIL ? detail + row * n * 2 : nullptr);
    if (lane == 0) {
      out[2 * row] = s.n;
      out[2 * row + 1] = (int64_t)s.t;
    }
    wave_sync_lds();
  }
}

// Algorithm 1 initialisation under the fitted model, one workgroup of 1024 threads, after
// the device checks of the queue (verdict to the header; a failed check ends the call):
// every request's latency alone (b = 1), a stable bitonic sort by (latency, id), the scores of the
// sorted and the input orders with maximum-size batches, t_ref.
__global__ void __launch_bounds__(1024) start_fit_kernel(DevFit f, QueuePtrs q, const uint32_t *thr2, int chains,
                                                          int iters, int64_t t_ref_user, SearchParams srch,
                                                          unsigned char *ws) {
  __shared__ uint4 req[1024];
  __shared__ uint64_t key_solo[1024];
  __shared__ uint16_t key_id[1024];
  __shared__ uint16_t ident[1024];
  const Plan plan = fit_plan_in_block(q, f);
  if (plan.status != 0) {
    if (threadIdx.x == 0) write_failed_header(ws, plan, f.n, chains, iters, f.policy, f.B);
    return;
  }
  if (threadIdx.x == 0) write_plan(ws, plan);
  fit_take_flags(f, plan.flags);
  const int n = f.n;
  const int tid = threadIdx.x;
  load_fit_requests(q, thr2, n, req);
  int np = 1;
  while (np < n) np <<= 1;
  if (tid < np) {
    if (tid < n) {
      const uint64_t l = q.in_len[tid], L = q.out_len[tid];
      key_solo[tid] = fit_prefill(f, 1, l) + fit_decode(f, 1, l, L);
      key_id[tid] = (uint16_t)tid;
      ident[tid] = (uint16_t)tid;
    } else {
      key_solo[tid] = ~0ull;
      key_id[tid] = 0xFFFFu;
    }
  }
  __syncthreads();
  for (int k = 2; k <= np; k <<= 1) {
    for (int j = k >> 1; j > 0; j >>= 1) {
      if (tid < np) {
        const int o = tid ^ j;
        if (o > tid) {
          const uint64_t a = key_solo[tid], b = key_solo[o];
          const uint16_t ia = key_id[tid], ib = key_id[o];
          const bool a_gt = a > b || (a == b && ia > ib);
          const bool up = (tid & k) == 0;
          if (a_gt == up) {
            key_solo[tid] = b;
            key_solo[o] = a;
            key_id[tid] = ib;
            key_id[o] = ia;
          }
        }
      }
      __syncthreads();
    }
  }
  if (tid < 64) {
    const Score sorted = replay_fit<false>(f, req, key_id, nullptr, nullptr);
    const Score input = replay_fit<false>(f, req, ident, nullptr, nullptr);
    const bool input_better = srch.objective ? obj_better<1>(input.n, input.t, sorted.n, sorted.t)
                                             : obj_better<0>(input.n, input.t, sorted.n, sorted.t);
    const bool use_input = !(srch.early_exit && sorted.n == n) && input_better;
    uint16_t *start = reinterpret_cast<uint16_t *>(ws + ws_off_start());
    for (int p = tid; p < n; p += 64) start[p] = use_input ? (uint16_t)p : key_id[p];
    if (tid == 0) {
      WsHeader *h = reinterpret_cast<WsHeader *>(ws);
      h->magic = kWsMagic;
      h->n = n;
      h->chains = chains;
      h->iters = iters;
      h->policy = f.policy;
      h->max_batch = f.B;
      h->objective = srch.objective;
      h->level_len = srch.level_len;
      h->early_exit = srch.early_exit;
      h->t_ref = t_ref_user > 0 ? t_ref_user : (input.t > 1 ? (int64_t)input.t : 1);
      h->start_n = use_input ? input.n : sorted.n;
      h->start_t = (int64_t)(use_input ? input.t : sorted.t);
      h->allmet = sorted.n == n ? 1 : 0;
      h->best_chain = -1;
      h->best_n = -1;
      h->best_t = -1;
    }
  }
}

// One wave per chain, four per workgroup; full replay per proposal. Fixed-size batches take
// swap / insert proposals (swap iff w0 < swap_thr); the batch-size search takes squeeze /
// delay / swap. Per-wave LDS: current and candidate orders and flags.
template <int OBJ>
__global__ void __launch_bounds__(256) anneal_fit_kernel(DevFit f, QueuePtrs q, const uint32_t *thr2, int chains,
                                                          int iters, double T0, double alpha, uint32_t key0,
                                                          uint32_t key1, uint64_t swap_thr, SearchParams srch,
                                                          unsigned char *ws) {
  extern __shared__ __align__(16) unsigned char lds[];
  if (!fit_gate_open(ws, f)) return;
  const int n = f.n, B = f.B;
  const bool search = f.policy == 2;
  uint4 *req = reinterpret_cast<uint4 *>(lds);
  const size_t pb = ((size_t)n * 2 + 15) & ~size_t(15), fb = ((size_t)n + 15) & ~size_t(15);
  const size_t per_wave = 2 * pb + 2 * fb;
  const int wave = uniform((int)(threadIdx.x >> 6));
  const int waves = blockDim.x >> 6;
  unsigned char *wb = lds + (((size_t)n * 16 + 15) & ~size_t(15)) + (size_t)wave * per_wave;
  uint16_t *cur = reinterpret_cast<uint16_t *>(wb);
  uint16_t *cand = reinterpret_cast<uint16_t *>(wb + pb);
  uint8_t *fcur = wb + 2 * pb, *fcand = wb + 2 * pb + fb;
  load_fit_requests(q, thr2, n, req);
  __syncthreads();
  const int chain = uniform((int)blockIdx.x * waves + wave);
  if (chain >= chains) return;
  const int lane = lane_id();
  const WsHeader *h = reinterpret_cast<const WsHeader *>(ws);
  const int64_t t_ref = h->t_ref, allmet = h->allmet;
  int64_t cn = h->start_n;
  uint64_t ct = (uint64_t)h->start_t;
  const uint16_t *start = reinterpret_cast<const uint16_t *>(ws + ws_off_start());
  const size_t stride = ws_perm_stride(n), fstride = ws_flag_stride(n);
  uint16_t *gbest = reinterpret_cast<uint16_t *>(ws + ws_off_best(n, chains)) + (size_t)chain * stride;
  uint16_t *gcur = reinterpret_cast<uint16_t *>(ws + ws_off_cur(n, chains)) + (size_t)chain * stride;
  uint8_t *gbest_f = ws + ws_off_best_starts(n, chains) + (size_t)chain * fstride;
  uint8_t *gcur_f = ws + ws_off_cur_starts(n, chains) + (size_t)chain * fstride;
  for (int p = lane; p < n; p += kWave) {
    const uint16_t v = start[p];
    const uint8_t fl = (uint8_t)(p % B == 0);
    cur[p] = v;
    fcur[p] = fl;
    gbest[p] = v;
    gbest_f[p] = fl;
  }
  wave_sync_lds();
  int64_t bn = cn, biter = -1, accepts = 0;
  uint64_t bt = ct, digest = kFnvOffset;
  Cooling cool{T0, alpha, srch.level_len, srch.level_len};
  SizedDraws ds;
  ProposalStream ps;
  const int iters_run = (srch.early_exit && allmet) ? 0 : iters;
  for (int k = 0; k < iters_run; ++k) {
    uint32_t w3;
    SizedMove mv;
    if (search) {
      if ((k & (kWave - 1)) == 0) ds.refill(k, lane, n, (uint32_t)chain, key0, key1);
      const uint32_t pk = ds.packed(k);
      w3 = ds.word3(k);
      mv = plan_move(fcur, n, B, (int)(pk >> 20), (int)(pk & 1023u), (int)((pk >> 10) & 1023u), lane);
    } else {
      if ((k & (kWave - 1)) == 0) ps.refill(k, lane, n, (uint32_t)chain, key0, key1, swap_thr, 0);
      const uint32_t pk = ps.packed(k);
      w3 = ps.word3(k);
      const int i = (int)(pk & 1023u), j = (int)((pk >> 10) & 1023u);
      // a fixed-size move: swap (op 2) or insert (from i to j, flags untouched)
      mv = SizedMove{true, ((pk >> 20) & 1u) ? 3 : 2, i, j, j, -1, -1};
    }
    if (mv.made) {
      for (int p = lane; p < n; p += kWave) {
        cand[p] = cur[p];
        fcand[p] = fcur[p];
      }
      wave_sync_lds();
      if (mv.op == 3)
        apply_move_lds(cand, 2, mv.i, mv.j, lane);
      else
        apply_sized_move(cand, fcand, mv, lane);
      const Score s = replay_fit<false>(f, req, cand, fcand, nullptr);
      if (obj_accept<OBJ>(cn, ct, s.n - cn, (int64_t)(s.t - ct), t_ref, cool.T, w3)) {
        uint16_t *tp = cur;
        cur = cand;
        cand = tp;
        uint8_t *tf = fcur;
        fcur = fcand;
        fcand = tf;
        cn = s.n;
        ct = s.t;
        ++accepts;
        digest = (digest ^ (uint64_t)k) * kFnvPrime;
        digest = (digest ^ (uint64_t)cn) * kFnvPrime;
        digest = (digest ^ ct) * kFnvPrime;
        if (obj_better<OBJ>(cn, ct, bn, bt)) {
          bn = cn;
          bt = ct;
          biter = k;
          for (int p = lane; p < n; p += kWave) {
            gbest[p] = cur[p];
            gbest_f[p] = fcur[p];
          }
        }
      }
    }
    cool.step();
  }
  for (int p = lane; p < n; p += kWave) {
    gcur[p] = cur[p];
    gcur_f[p] = fcur[p];
  }
  if (lane == 0) write_record(ws, n, chain, cn, ct, bn, bt, biter, accepts, digest, allmet);
}

}  // namespace sa
