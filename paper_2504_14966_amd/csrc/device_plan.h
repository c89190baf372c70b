// Device-side checks of a request queue: whether every entry is valid, whether the int64
// clock and objective are safe for this queue and model, and which integer widths hold,
// which picks the kernel of a call. The calls run these checks on the GPU instead of
// copying the queue to the host, so that nothing blocks.
//
// Every bound is an exact integer (saturating at 2^64 - 1, products formed in 128 bits),
// compared against the limits each kernel is written for:
//   range: the timeline of any order ends before every prefill plus, per decode step (at
//     most the sum of output lengths), the cost of a full batch of the longest contexts;
//     n times that, and t_ref (n + 1) plus it, stay below 2^62 (and for the ratio
//     objective n + 1 times it too);
//   widths: see plan_decide.
// An annealing call's first kernel (the one that forms the start order) forms the verdict
// and writes it to the workspace header, where every later kernel of the call reads it; the
// evaluation calls have no workspace, so every workgroup forms it (plan_in_block) from the
// queue it stages anyway.
#pragma once
#include "device_common.h"

namespace sa {

constexpr int32_t kPlanEInval = -1;  // SCHED_EINVAL
constexpr int32_t kPlanERange = -3;  // SCHED_ERANGE
constexpr uint32_t kThrMax = 0xFFFFFFFEu;

__host__ __device__ __forceinline__ uint64_t sat_add(uint64_t a, uint64_t b) {
  const uint64_t s = a + b;
  return s < a ? ~0ull : s;
}
__host__ __device__ __forceinline__ uint64_t sat_mul(uint64_t a, uint64_t b) {
  const unsigned __int128 p = (unsigned __int128)a * b;
  return (uint64_t)(p >> 64) ? ~0ull : (uint64_t)p;
}

// Coefficients of the fitted model (Latency Predictor: per-request prefill and decode with
// the batch-size interaction terms), for the checks of the fitted-model calls.
struct FitCoef {
  uint64_t ap, bp, cp, dp, ad, bd, cd, dd;
};

// Time of one request of l input and L output tokens in a batch of b under the fitted model:
// ap b l + bp b + cp l + dp + L (bd b + dd) + (ad b + cd) (L l + L (L + 1) / 2), saturating.
__host__ __device__ __forceinline__ uint64_t fit_member_time(const FitCoef &c, uint64_t b, uint64_t l, uint64_t L) {
  uint64_t t = sat_mul(sat_mul(c.ap, b), l);
  t = sat_add(t, sat_mul(c.bp, b));
  t = sat_add(t, sat_mul(c.cp, l));
  t = sat_add(t, c.dp);
  t = sat_add(t, sat_mul(L, sat_add(sat_mul(c.bd, b), c.dd)));
  return sat_add(t, sat_mul(sat_add(sat_mul(c.ad, b), c.cd), L * l + L * (L + 1) / 2));
}

// What the checks need from the queue, reduced over all of it.
struct QueueStats {
  uint32_t bad;        // some entry has l_out = 0, a kind above max_kind or a threshold above kThrMax
  uint32_t lmax, Lmax;  // longest input, longest output
  uint32_t pad;
  uint64_t slin, sL, sctx;  // sums of l_in, of l_out, of l_out l_in + l_out (l_out + 1) / 2
  uint64_t fit_max, fit_sum;  // fitted model: largest and summed member time in a batch of min(n, B)
};

struct Plan {
  int32_t status;   // 0 or kPlanEInval / kPlanERange
  uint32_t flags;   // kFlag* widths that hold
  int32_t selected;  // the candidate that runs, -1 when status != 0
};

// The checks on the reduced statistics. fit: the fitted model's coefficients or null.
__host__ __device__ inline Plan plan_decide(const QueueStats &s, int n_, int B, int ratio, int64_t t_ref,
                                            uint64_t p0, uint64_t p1, uint64_t d0, uint64_t d1, uint64_t d2,
                                            const FitCoef *fit, const Gate &gate) {
  Plan p{0, 0u, -1};
  if (s.bad) {
    p.status = kPlanEInval;
    return p;
  }
  const uint64_t n = (uint64_t)n_, b = (uint64_t)(n_ < B ? n_ : B);
  const uint64_t lim62 = 1ull << 62, two32 = 1ull << 32, two24 = 1ull << 24, two57 = 1ull << 57;
  const uint64_t lmax = s.lmax, Lmax = s.Lmax;
  uint64_t end;  // bound on the end of the timeline of any order
  if (fit) {
    // a member's time grows with its batch size and a batch lasts at most the sum of its
    // members' times, so the sum of the times in a batch of min(n, B) bounds the timeline
    end = s.fit_sum;
    if (end < two57) p.flags |= kFlagFitWindows;
    if (s.fit_max < two32 - 1) p.flags |= kFlagFitMember32;
  } else {
    const uint64_t pre = sat_add(sat_mul(n, p0), sat_mul(p1, s.slin));  // every prefill
    const uint64_t step = sat_add(sat_add(d0, sat_mul(d1, b)), sat_mul(sat_mul(d2, b), lmax + Lmax));
    end = sat_add(pre, sat_mul(s.sL, step));
    // continuous event arithmetic in 32 bits: a group prefill, the running context sum,
    // one decode step and d2 b
    const uint64_t pf1 = sat_add(p0, sat_mul(p1, lmax));
    const uint64_t cmax = b * (lmax + Lmax);
    const uint64_t x = sat_add(sat_add(d0, sat_mul(d1, b)), sat_mul(d2, cmax));
    const bool narrow_prefill = sat_mul(pf1, b) < two32 && cmax < two32 && x < two32 && sat_mul(d2, b) < two32;
    // list scheduling: keys (finish step << 10 | position) and prefill prefix sums in 32 bits
    const bool list = s.sL < (1ull << 22) && pre < two32;
    // every time on a timeline of any order or layout: the prefills, plus over the decode
    // steps (at most sum l_out) their d0 + d1 b terms (which add up to at most (d0 + d1)
    // sum l_out) and d2 C terms (which add up to d2 sum (l_out l_in + l_out (l_out + 1) / 2))
    const uint64_t tl = sat_add(sat_add(pre, sat_mul(sat_add(d0, d1), s.sL)), sat_mul(d2, s.sctx));
    if (narrow_prefill) {
      p.flags |= kFlagNarrowPrefill;
      if (list) {
        p.flags |= kFlagListSched;
        if (tl < two32) p.flags |= kFlagNarrowTime;
      }
    }
    if (end < two57) p.flags |= kFlagWindows;
    // static delta widths: every finish offset within a batch below 2^32 - 1 (at most B
    // prefills, L_max d0 and B times a member's decode terms), doubled pair costs
    // mu (e + d2 mu) with 24-bit factors, e = 2 (d1 + d2 l_in) + d2
    const uint64_t tri = Lmax * (Lmax + 1) / 2;
    const uint64_t fmax =
        sat_add(sat_add(sat_mul(b, pf1), sat_mul(Lmax, d0)),
                sat_mul(b, sat_add(sat_mul(d1, Lmax), sat_mul(d2, lmax * Lmax + tri))));
    const uint64_t emax = sat_add(sat_mul(2, sat_add(d1, sat_mul(d2, lmax))), d2);
    const uint64_t inner = sat_add(emax, sat_mul(d2, Lmax));
    const bool snarrow = fmax < two32 - 1 && inner < two24 && d2 < two24 && sat_mul(b * Lmax, inner) < two32 &&
                         d0 < two24;
    if (snarrow) {
      p.flags |= kFlagStaticNarrow;
      if (tl < two32 - 2) p.flags |= kFlagTime32;
    }
  }
  const uint64_t tsum = sat_mul(end, n);
  const uint64_t tref = t_ref > 0 ? (uint64_t)t_ref : tsum;
  if (!(tsum < lim62) || !(sat_add(sat_mul(tref, n + 1), tsum) < lim62) ||
      (ratio && !(sat_mul(tsum, n + 1) < lim62))) {
    p.status = kPlanERange;
    p.flags = 0u;
    return p;
  }
  return p;
}

// The first candidate whose needs hold (the loop is unrolled so that the candidate list is
// only ever indexed by constants and the model it travels in stays in registers).
__host__ __device__ inline int32_t plan_select(const Gate &g, uint32_t flags) {
  int32_t sel = -1;
#pragma unroll
  for (int c = 3; c >= 0; --c)
    if (c < g.count && (g.need[c] & flags) == g.need[c]) sel = c;
  return sel;
}

// Static LDS the checks take in a workgroup (on top of a kernel's dynamic LDS).
constexpr size_t kCheckLdsBytes = 16 * 8 * 8;

// Statistics of the queue reduced by the whole workgroup (every thread must call it; one
// barrier inside). fit: coefficients of the fitted model or null.
__device__ QueueStats block_queue_stats(const QueuePtrs &q, int n, int B, int max_kind, const FitCoef *fit) {
  __shared__ uint64_t red[16][8];
  static_assert(sizeof(red) == kCheckLdsBytes, "static LDS of the checks");
  uint32_t bad = 0, lmax = 0, Lmax = 0;
  uint64_t slin = 0, sL = 0, sctx = 0, fmax = 0, fsum = 0;
  const uint64_t b = (uint64_t)(n < B ? n : B);
  for (int r = threadIdx.x; r < n; r += blockDim.x) {
    const uint32_t l = q.in_len[r], L = q.out_len[r], kind = q.kind[r], thr = q.thr[r];
    bad |= (L < 1u || kind > (uint32_t)max_kind || thr > kThrMax) ? 1u : 0u;
    lmax = max(lmax, l);
    Lmax = max(Lmax, L);
    slin += l;
    sL += L;
    sctx += (uint64_t)L * l + (uint64_t)L * (L + 1) / 2;
    if (fit) {
      const uint64_t t = fit_member_time(*fit, b, l, L);
      fmax = fmax > t ? fmax : t;
      fsum = sat_add(fsum, t);
    }
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) {
    bad |= (uint32_t)__shfl_xor((int)bad, o);
    lmax = max(lmax, (uint32_t)__shfl_xor((int)lmax, o));
    Lmax = max(Lmax, (uint32_t)__shfl_xor((int)Lmax, o));
    slin += __shfl_xor(slin, o);
    sL += __shfl_xor(sL, o);
    sctx += __shfl_xor(sctx, o);
    const uint64_t fm = __shfl_xor(fmax, o), fs = __shfl_xor(fsum, o);
    fmax = fmax > fm ? fmax : fm;
    fsum = sat_add(fsum, fs);
  }
  const int wave = (int)(threadIdx.x >> 6), waves = (int)((blockDim.x + 63) >> 6);
  if ((threadIdx.x & 63u) == 0) {
    red[wave][0] = bad;
    red[wave][1] = lmax;
    red[wave][2] = Lmax;
    red[wave][3] = slin;
    red[wave][4] = sL;
    red[wave][5] = sctx;
    red[wave][6] = fmax;
    red[wave][7] = fsum;
  }
  __syncthreads();
  QueueStats s{0u, 0u, 0u, 0u, 0ull, 0ull, 0ull, 0ull, 0ull};
  for (int w = 0; w < waves; ++w) {
    s.bad |= (uint32_t)red[w][0];
    s.lmax = max(s.lmax, (uint32_t)red[w][1]);
    s.Lmax = max(s.Lmax, (uint32_t)red[w][2]);
    s.slin += red[w][3];
    s.sL += red[w][4];
    s.sctx += red[w][5];
    s.fit_max = s.fit_max > red[w][6] ? s.fit_max : red[w][6];
    s.fit_sum = sat_add(s.fit_sum, red[w][7]);
  }
  return s;
}

// The plan of an integer-model call, formed by the whole workgroup.
__device__ __forceinline__ Plan plan_in_block(const QueuePtrs &q, const DevModel &m) {
  const QueueStats s = block_queue_stats(q, m.n, m.B, m.max_kind, nullptr);
  Plan p = plan_decide(s, m.n, m.B, m.ratio, m.t_ref, m.p0, m.p1, m.d0, m.d1, m.d2, nullptr, m.gate);
  if (p.status == 0) p.selected = plan_select(m.gate, p.flags);
  return p;
}

// Reads the plan a call's plan kernel left in the workspace header: true when this launch is
// the selected candidate, with the allowed check flags added to `flags`.
__device__ __forceinline__ bool gate_open(const unsigned char *ws, const Gate &g, int32_t &flags) {
  const WsHeader *h = reinterpret_cast<const WsHeader *>(ws);
  if (h->plan_selected != (int64_t)g.self) return false;
  flags |= (int32_t)((uint32_t)h->plan_flags & g.allow);
  return true;
}
__device__ __forceinline__ bool plan_ok(const unsigned char *ws) {
  return reinterpret_cast<const WsHeader *>(ws)->plan_status == 0;
}

// Launches that run whenever the checks passed (start orders, reductions): the allowed
// check flags are added to `flags`.
__device__ __forceinline__ bool gate_status(const unsigned char *ws, const Gate &g, int32_t &flags) {
  const WsHeader *h = reinterpret_cast<const WsHeader *>(ws);
  if (h->plan_status != 0) return false;
  flags |= (int32_t)((uint32_t)h->plan_flags & g.allow);
  return true;
}

// Every row of an evaluation call whose queue failed the checks reads (-2, code).
__device__ __forceinline__ void error_rows(int64_t rows, int32_t status, int64_t *out) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r < rows; r += stride) {
    out[2 * r] = -2;
    out[2 * r + 1] = status;
  }
}

// Evaluation calls have no workspace. The first candidate launched forms the verdict in
// every workgroup: on a failed check it writes the error rows; when another candidate is
// selected, its workgroup 0 leaves the verdict in row 0 of the output as a marker
// (kEvalMarker - selected, flags) and no row is replayed. A later candidate reads the marker
// and, when it is the one selected, replays rows 1 .. rows - 1; the fix-up launch after
// every candidate (self == kEvalFixup) finds the marker still there and replays row 0. Row
// 0 is written by no candidate that reads it, so no workgroup can see it overwritten.
constexpr int64_t kEvalMarker = -16;
constexpr int32_t kEvalFixup = -2;

struct EvalRows {
  int64_t begin, end;  // rows this launch replays (none when end <= begin)
};

// The launch's rows, with the allowed flags of the verdict added to `flags`. plan: forms the
// verdict (called by the first candidate only).
template <class PlanFn>
__device__ __forceinline__ EvalRows eval_rows_of(PlanFn plan, const Gate &g, int64_t rows, int64_t *out,
                                                 uint32_t &flags) {
  if (g.self != 0) {
    const int64_t mark = out[0];
    const bool mine = g.self == kEvalFixup ? mark <= kEvalMarker : mark == kEvalMarker - g.self;
    if (!mine) return EvalRows{0, 0};
    flags |= (uint32_t)out[1] & g.allow;
    return g.self == kEvalFixup ? EvalRows{0, 1} : EvalRows{1, rows};
  }
  const Plan p = plan();
  if (p.status != 0) {
    error_rows(rows, p.status, out);
    return EvalRows{0, 0};
  }
  if (p.selected != 0) {
    if (blockIdx.x == 0 && threadIdx.x == 0) {
      out[0] = kEvalMarker - p.selected;
      out[1] = (int64_t)p.flags;
    }
    return EvalRows{0, 0};
  }
  flags |= p.flags & g.allow;
  return EvalRows{0, rows};
}

__device__ __forceinline__ EvalRows eval_gate(const QueuePtrs &q, DevModel &m, int64_t rows, int64_t *out) {
  uint32_t f = 0u;
  const EvalRows r = eval_rows_of([&]() { return plan_in_block(q, m); }, m.gate, rows, out, f);
  m.flags |= (int32_t)f;
  return r;
}

// The verdict into a workspace header (thread 0 of the checking workgroup).
__device__ __forceinline__ void write_plan(unsigned char *ws, const Plan &p) {
  WsHeader *h = reinterpret_cast<WsHeader *>(ws);
  h->plan_status = p.status;
  h->plan_flags = p.flags;
  h->plan_selected = p.selected;
}

// A call whose queue failed the checks still leaves a header the readouts can use: its
// sizes, no winner, the verdict.
__device__ __forceinline__ void write_failed_header(unsigned char *ws, const Plan &p, int n, int chains, int iters,
                                                    int policy, int B) {
  WsHeader *h = reinterpret_cast<WsHeader *>(ws);
  h->magic = kWsMagic;
  h->n = n;
  h->chains = chains;
  h->iters = iters;
  h->policy = policy;
  h->max_batch = B;
  h->best_chain = -1;
  h->best_n = -1;
  h->best_t = -1;
  write_plan(ws, p);
}

}  // namespace sa