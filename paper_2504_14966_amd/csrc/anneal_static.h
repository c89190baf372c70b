// Annealing chains under static admission with delta re-simulation (gfx950, wave64).
//
// Why a delta works. Under static admission the batch of position p is p / B and a
// batch's duration does not depend on when it starts (waiting-time equation of the
// Problem Formulation). A swap of positions in batches a < c, or an insert that moves
// one request from batch a to batch c (or back), changes the membership of batches
// a..c by exactly one request each: one request leaves (o) and one joins (e). Every
// other batch keeps its members and only its start time shifts by the change in
// duration of the changed batches before it. A move inside one batch changes nothing.
//
// State per chain (LDS): the order (u16 per position), every request's finish offset F
// within its batch including the prefill (u32, indexed by request id), and one record
// per batch: start S, sum of F, prefill P, duration D = max F, SLO-met count at S, and
// two bounds on S inside which no member's SLO flag changes (see Slack below).
//
// For a changed batch with prefill P -> P' = P + pf(e) - pf(o), a staying member m gets
//   F'_m = F_m + (P' - P) + (w(e, m) - w(o, m)) / 2,
// and the newcomer F'_e = P' + L_e * d0 + sum over the new members j of w(j, e) / 2, where
//   w(j, m) = mu * (e_j + d2 * mu),  mu = min(L_j, L_m),  e_j = 2 (d1 + d2 l_j) + d2,
// is twice the per-token decode cost that member j adds to m's decode iterations
// (d1 * mu + d2 * (l_j mu + mu (mu + 1) / 2)). Both factors stay below 2^24, so each w is
// one 24-bit multiply-add and one 24-bit multiply.
//
// The candidate objective is n + (met-count changes) and t + (size * start shift summed
// over later batches) + (change of sum F of the changed batches). A batch whose members
// are unchanged and whose new start stays inside its two bounds keeps its met count: it
// costs one lane of a batch-parallel check. Only batches that cross a bound are recounted
// member by member.
//
// Candidate F values are written speculatively (acceptance is the common case); a
// rejected proposal restores them with the reverse update (o and e exchanged). Candidate
// batch records go to a second array that is copied on accept.
//
// Lane layout: a batch occupies Bp = 2^LG lanes (B <= Bp), G = 64 / Bp batches per row.
// Widths: F, P, D, w and slacks are u32 (the device check keeps every finish offset and 2w
// below 2^32 and the multiply-add operands below 2^24); starts, sums, objective are u64.
#pragma once
#include "device_common.h"
#include "device_cont.h"
#include "device_plan.h"
#include "device_replay.h"
#include "device_rng.h"

namespace sa {

struct alignas(16) BatchRec {
  uint64_t S;    // start time
  uint64_t SF;   // sum of member finish offsets
  uint32_t P;    // prefill of the batch
  uint32_t D;    // duration = max finish offset
  uint32_t cnt;  // members meeting their SLO when the batch starts at S
  uint32_t A;    // every member keeps its SLO flag while Bv <= start <= A
  uint32_t Bv;
  uint32_t pad[3];
};

struct StaticParams {
  uint32_t d0, d2;
  uint64_t bmagic;  // floor(2^32 / B) + 1 (2^32 + 1 for B = 1): p / B == (p * bmagic) >> 32 for p < 2^16
};

__device__ __forceinline__ uint32_t div_b(uint32_t p, uint64_t bmagic) {
  return (uint32_t)(((uint64_t)p * bmagic) >> 32);
}

// Request record in LDS: x = l_in | l_out << 16, y = threshold, z = kind | e << 2, w = prefill.
struct Req {
  uint32_t L, thr, kind, e, pf;
};
__device__ __forceinline__ Req load_req(const uint4 *req, int r) {
  const uint4 v = req[r];
  return Req{v.x >> 16, v.y, v.z & 3u, v.z >> 2, v.w};
}

// v_mad_u32_u24: a * b + c for a, b below 2^24 (the compiler would otherwise fuse the
// multiply-add into a 64-bit v_mad_u64_u32)
__device__ __forceinline__ uint32_t mad24_v(uint32_t a, uint32_t b, uint32_t c) {
  uint32_t d;
  asm("v_mad_u32_u24 %0, %1, %2, %3" : "=v"(d) : "v"(a), "v"(b), "v"(c));
  return d;
}

// twice the decode cost member j (output L_j, e_j) adds to a member with output Lm
__device__ __forceinline__ uint32_t w2(uint32_t Lj, uint32_t ej, uint32_t Lm, uint32_t d2) {
  const uint32_t mu = min(Lj, Lm);
  return mad24_v(mu, mad24_v(d2, mu, ej), 0u);
}

// SLO flag of a member as a function of its batch start S: TPOT does not depend on S;
// TTFT (offset P) and end-to-end (offset F) are met iff S <= thr - offset =: slack.
// For TPOT requests the record's threshold field holds min(thr * l_out, 2^32 - 1): the
// decode time F - P is below 2^32 - 1, so the test (F - P) <= thr * l_out is one compare.
struct Slack {
  bool always, never;
  uint32_t s;
};
__device__ __forceinline__ Slack slack_of(uint32_t kind, uint32_t thr, uint32_t L, uint32_t P, uint32_t F) {
  const bool tpot = kind == 1;
  const bool tpot_ok = F - P <= thr;
  const uint32_t off = kind == 0 ? P : F;
  const bool late = off > thr;
  return Slack{tpot && tpot_ok, tpot ? !tpot_ok : late, thr - off};
}
__device__ __forceinline__ bool slack_met(const Slack &x, uint64_t S) { return x.always || (!x.never && S <= x.s); }

// Cross-lane primitives on gfx950 DPP: quad_perm [1,0,3,2] and [2,3,0,1] pair lanes at
// distance 1 and 2, row_half_mirror pairs the two quads of each half-row and row_mirror
// the two half-rows, so four DPP steps all-reduce a 16-lane row; whole-wave results come
// from v_readlane of the four row leaders into scalar registers.
template <int CTRL>
__device__ __forceinline__ uint32_t dpp(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, true);
}
// quad_perm and the two mirrors read a valid lane for every lane, so no fill value is used
constexpr int kQuadXor1 = 0xB1, kQuadXor2 = 0x4E, kRowHalfMirror = 0x141, kRowMirror = 0x140;

__device__ __forceinline__ uint32_t readlane(uint32_t v, int l) { return (uint32_t)__builtin_amdgcn_readlane((int)v, l); }
// v_writelane of a wave-uniform value into lane k (lane select in m0)
__device__ __forceinline__ uint32_t wlane_m0(uint32_t v, int k, uint32_t old) {
  asm volatile("v_writelane_b32 %0, %1, m0" : "=v"(old) : "s"(v), "{m0}"(k), "0"(old));
  return old;
}

struct OpAdd {
  static constexpr uint32_t identity = 0u;
  __device__ static __forceinline__ uint32_t f(uint32_t a, uint32_t b) { return a + b; }
};
struct OpMax {
  static constexpr uint32_t identity = 0u;
  __device__ static __forceinline__ uint32_t f(uint32_t a, uint32_t b) { return max(a, b); }
};
struct OpMin {
  static constexpr uint32_t identity = 0xFFFFFFFFu;
  __device__ static __forceinline__ uint32_t f(uint32_t a, uint32_t b) { return min(a, b); }
};

template <int LG>
struct Seg {
  static constexpr int Bp = 1 << LG;
  // all-reduce over each segment of Bp lanes; every lane receives its segment's result.
  // Lanes outside any batch must hold the identity of Op.
  template <class Op>
  __device__ static __forceinline__ uint32_t all(uint32_t v, int lane) {
    if constexpr (LG >= 1) v = Op::f(v, dpp<kQuadXor1>(v));
    if constexpr (LG >= 2) v = Op::f(v, dpp<kQuadXor2>(v));
    if constexpr (LG >= 3) v = Op::f(v, dpp<kRowHalfMirror>(v));
    if constexpr (LG >= 4) v = Op::f(v, dpp<kRowMirror>(v));
    if constexpr (LG >= 5) {
      // rows 1 and 3 combine the last lane of rows 0 and 2: each 32-lane half is reduced
      // in its last row
      v = Op::f(v, (uint32_t)__builtin_amdgcn_update_dpp((int)Op::identity, (int)v, 0x142, 0xA, 0xF, false));
    }
    if constexpr (LG == 5) {
      v = lane < 32 ? readlane(v, 31) : readlane(v, 63);
    }
    if constexpr (LG == 6) {
      v = Op::f(v, (uint32_t)__builtin_amdgcn_update_dpp((int)Op::identity, (int)v, 0x143, 0xC, 0xF, false));
      v = readlane(v, 63);
    }
    return v;
  }
  // the same reductions taken two or three at a time, step by step, so that the DPP steps
  // of one fill the wait states of the other
  static constexpr int kSteps = LG;  // quad, quad, half-row, row, then one or two row broadcasts
  template <class Op>
  __device__ static __forceinline__ uint32_t step(uint32_t v, int s) {
    switch (s) {
      case 0: return Op::f(v, dpp<kQuadXor1>(v));
      case 1: return Op::f(v, dpp<kQuadXor2>(v));
      case 2: return Op::f(v, dpp<kRowHalfMirror>(v));
      case 3: return Op::f(v, dpp<kRowMirror>(v));
      case 4: return Op::f(v, (uint32_t)__builtin_amdgcn_update_dpp((int)Op::identity, (int)v, 0x142, 0xA, 0xF, false));
      default: return Op::f(v, (uint32_t)__builtin_amdgcn_update_dpp((int)Op::identity, (int)v, 0x143, 0xC, 0xF, false));
    }
  }
  __device__ static __forceinline__ uint32_t finish(uint32_t v, int lane) {
    if constexpr (LG == 5) return lane < 32 ? readlane(v, 31) : readlane(v, 63);
    if constexpr (LG == 6) return readlane(v, 63);
    return v;
  }
  template <class O1, class O2>
  __device__ static __forceinline__ void all2(uint32_t &a, uint32_t &b, int lane) {
#pragma unroll
    for (int s = 0; s < kSteps; ++s) {
      a = step<O1>(a, s);
      b = step<O2>(b, s);
    }
    a = finish(a, lane);
    b = finish(b, lane);
  }
  template <class O1, class O2, class O3>
  __device__ static __forceinline__ void all3(uint32_t &a, uint32_t &b, uint32_t &c, int lane) {
#pragma unroll
    for (int s = 0; s < kSteps; ++s) {
      a = step<O1>(a, s);
      b = step<O2>(b, s);
      c = step<O3>(c, s);
    }
    a = finish(a, lane);
    b = finish(b, lane);
    c = finish(c, lane);
  }
  template <class O1, class O2, class O3, class O4>
  __device__ static __forceinline__ void all4(uint32_t &a, uint32_t &b, uint32_t &c, uint32_t &d, int lane) {
#pragma unroll
    for (int s = 0; s < kSteps; ++s) {
      a = step<O1>(a, s);
      b = step<O2>(b, s);
      c = step<O3>(c, s);
      d = step<O4>(d, s);
    }
    a = finish(a, lane);
    b = finish(b, lane);
    c = finish(c, lane);
    d = finish(d, lane);
  }
  // exact sum of 32-bit values as two 16-bit-half sums (each below 2^22)
  __device__ static __forceinline__ uint64_t sum_wide(uint32_t v, int lane) {
    const uint32_t lo = all<OpAdd>(v & 0xFFFFu, lane), hi = all<OpAdd>(v >> 16, lane);
    return (uint64_t)lo + ((uint64_t)hi << 16);
  }
  // segment-uniform v: exclusive prefix over the segments of the row, and the row total
  __device__ static __forceinline__ void scan(int64_t v, int lane, int64_t &excl, int64_t &total) {
    if constexpr (LG == 6) {
      excl = 0;
      total = v;
    } else if constexpr (LG >= 4) {
      int64_t s[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const uint32_t lo = readlane((uint32_t)(uint64_t)v, u * 16), hi = readlane((uint32_t)((uint64_t)v >> 32), u * 16);
        s[u] = (int64_t)(((uint64_t)hi << 32) | lo);
      }
      if constexpr (LG == 5) {
        total = s[0] + s[2];
        excl = lane < 32 ? 0 : s[0];
      } else {
        total = s[0] + s[1] + s[2] + s[3];
        const int g = lane >> 4;
        excl = g == 0 ? 0 : (g == 1 ? s[0] : (g == 2 ? s[0] + s[1] : s[0] + s[1] + s[2]));
      }
    } else {
      int64_t x = (lane & (Bp - 1)) == 0 ? v : 0;
#pragma unroll
      for (int o = Bp; o < kWave; o <<= 1) {
        const int64_t y = __shfl_up(x, o);
        if (lane >= o) x += y;
      }
      excl = __shfl(x, lane & ~(Bp - 1)) - v;
      total = __shfl(x, kWave - Bp);
    }
  }
  __device__ static __forceinline__ int count(bool p, int seg) {
    uint64_t m = __ballot(p);
    if (Bp < kWave) m = (m >> (seg << LG)) & ((1ull << (Bp & 63)) - 1ull);
    return __popcll(m);
  }
  // sum over lanes of a value that only segment leaders (lanes 0, Bp, 2Bp, ...) hold
  __device__ static __forceinline__ int64_t leader_sum(int64_t v) {
    if constexpr (LG >= 4) {
      int64_t s = 0;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        if (LG == 6 && u > 0) break;
        if (LG == 5 && (u & 1)) continue;
        const uint32_t lo = readlane((uint32_t)(uint64_t)v, u * 16), hi = readlane((uint32_t)((uint64_t)v >> 32), u * 16);
        s += (int64_t)(((uint64_t)hi << 32) | lo);
      }
      return s;
    } else {
      return (int64_t)wave_sum_u64((uint64_t)v);
    }
  }
};

// A proposal: move type (1 swap, 2 insert), positions, changed batch range [a, c].
struct Move {
  int type, i, j, a, c;
  __device__ __forceinline__ bool changes(int k) const { return k >= a && k <= c && (type == 2 || k == a || k == c); }
};

template <int LG>
struct StaticChain {
  const uint4 *req;
  uint16_t *perm;
  uint32_t *F;
  BatchRec *cur;
  BatchRec *cand;
  StaticParams sp;
  int N, B, M, R;  // requests, batch size, batches, rows
  int lane, seg, mm;
  static constexpr int Bp = 1 << LG;
  static constexpr int G = kWave >> LG;

  __device__ __forceinline__ int batch_size(int k) const { return min(B, N - k * B); }
  // requests in batches [k0, k1)
  __device__ __forceinline__ int64_t requests_in(int k0, int k1) const {
    return k1 <= k0 ? 0 : (int64_t)min(N, k1 * B) - (int64_t)k0 * B;
  }

  // Member-level pass over one row. Batches below `a` are left alone; changed batches get
  // candidate F (written speculatively); every other live batch is recounted at its start
  // moved by base_shift plus the duration changes of the changed batches before it in the
  // row. Writes candidate records and adds the met-count change of the row's batches to
  // dn_l, and (with add_dt) their latency change to dt_l (segment leaders). Returns the
  // row's total duration change.
  __device__ int64_t row_pass(int row, const Move &mv, int64_t base_shift, bool add_dt, int64_t &dn_l,
                              int64_t &dt_l) {
    const int k = row * G + seg;
    const int q = k * B + mm;
    const bool valid = mm < B && q < N;
    const bool seg_live = k < M && k >= mv.a;                // uniform per segment
    const bool seg_changed = seg_live && mv.changes(k);
    const int k0 = row * G, k1 = min(row * G + G - 1, M - 1);
    const bool row_changed = mv.type == 2 ? (mv.a <= k1 && mv.c >= k0)
                                          : ((mv.a >= k0 && mv.a <= k1) || (mv.c >= k0 && mv.c <= k1));
    const BatchRec br = cur[min(k, M - 1)];
    const int r = valid ? (int)perm[min(q, N - 1)] : N;  // lanes outside a batch use the spare slot N
    Req rq = load_req(req, r);
    uint32_t Fn = F[r];  // the spare slot N reads as 0 for lanes outside a batch
    uint32_t Pn = br.P, Dn = br.D;
    uint64_t SFn = br.SF;
    if (row_changed) {
      int o = 0, e = 0;
      out_in(seg_changed ? k : mv.a, mv, o, e);
      const Req ro = load_req(req, o), re = load_req(req, e);
      const uint32_t Pc = br.P + re.pf - ro.pf;
      const bool is_out = seg_changed && r == o;
      const int rn = is_out ? e : r;
      if (is_out) rq = re;
      // newcomer: prefill, its own decode steps and what every new member adds to them
      const uint32_t te = (seg_changed && valid) ? w2(rq.L, rq.e, re.L, sp.d2) : 0u;
      const uint32_t Fe = Pc + __umul24(re.L, sp.d0) + (Seg<LG>::template all<OpAdd>(te, lane) >> 1);
      const int32_t dw = (int32_t)(w2(re.L, re.e, rq.L, sp.d2) - w2(ro.L, ro.e, rq.L, sp.d2));
      const uint32_t Fc = is_out ? Fe : Fn + (Pc - br.P) + (uint32_t)(dw >> 1);
      if (seg_changed) {
        Fn = valid ? Fc : 0u;
        Pn = Pc;
      }
      if (seg_changed && valid) F[rn] = Fc;
      uint32_t Dm = Fn, SFlo = Fn & 0xFFFFu, SFhi = Fn >> 16;
      Seg<LG>::template all3<OpMax, OpAdd, OpAdd>(Dm, SFlo, SFhi, lane);
      const uint64_t SFm = (uint64_t)SFlo + ((uint64_t)SFhi << 16);
      if (seg_changed) {
        Dn = Dm;
        SFn = SFm;
      }
    }
    const int64_t dlt = seg_changed ? (int64_t)Dn - (int64_t)br.D : 0;
    int64_t excl, total;
    Seg<LG>::scan(dlt, lane, excl, total);
    const int64_t shift = base_shift + excl;
    const uint64_t Sn = br.S + (uint64_t)shift;
    const bool in_range = valid && seg_live;
    const Slack x = slack_of(rq.kind, rq.thr, rq.L, Pn, Fn);
    const bool met = in_range && slack_met(x, Sn);
    const int cnt = Seg<LG>::count(met, seg);
    uint32_t A = (in_range && met && !x.always) ? x.s : 0xFFFFFFFFu;
    uint32_t Bv = (in_range && !met && !x.never) ? x.s + 1u : 0u;
    Seg<LG>::template all2<OpMin, OpMax>(A, Bv, lane);
    if (mm == 0 && seg_live) {
      dn_l += (int64_t)cnt - (int64_t)br.cnt;
      if (add_dt) dt_l += (int64_t)batch_size(k) * shift + (int64_t)(SFn - br.SF);
      cand[k] = BatchRec{Sn, SFn, Pn, Dn, (uint32_t)cnt, A, Bv, {0, 0, 0}};
    }
    return total;
  }

  // Full evaluation of the current order: F of every request and every batch record.
  __device__ Score init() {
    uint64_t carry = 0, tl = 0;
    int64_t nmet = 0;
    if (lane == 0) F[N] = 0u;  // spare slot read by lanes outside a batch
    for (int row = 0; row < R; ++row) {
      const int k = row * G + seg;
      const int q = k * B + mm;
      const bool valid = mm < B && q < N;
      Req rq{0, 0, 0, 0, 0};
      int r = 0;
      if (valid) {
        r = perm[q];
        rq = load_req(req, r);
      }
      // pairwise closed form over the members of this lane's batch
      uint32_t P = 0, acc = 0;
      for (int jj = 0; jj < B; ++jj) {
        const int qj = k * B + jj;
        if (k < M && qj < N) {
          const Req o = load_req(req, perm[qj]);
          P += o.pf;
          acc += w2(o.L, o.e, rq.L, sp.d2);
        }
      }
      const uint32_t Fv = valid ? P + __umul24(rq.L, sp.d0) + (acc >> 1) : 0u;
      if (valid) F[r] = Fv;
      const uint32_t D = Seg<LG>::template all<OpMax>(Fv, lane);
      const uint64_t SF = Seg<LG>::sum_wide(Fv, lane);
      int64_t excl, total;
      Seg<LG>::scan(k < M ? (int64_t)D : 0, lane, excl, total);
      const uint64_t S = carry + (uint64_t)excl;
      const Slack x = slack_of(rq.kind, rq.thr, rq.L, P, Fv);
      const bool met = valid && slack_met(x, S);
      const int cnt = Seg<LG>::count(met, seg);
      const uint32_t A = Seg<LG>::template all<OpMin>((valid && met && !x.always) ? x.s : 0xFFFFFFFFu, lane);
      const uint32_t Bv = Seg<LG>::template all<OpMax>((valid && !met && !x.never) ? x.s + 1u : 0u, lane);
      if (mm == 0 && k < M) {
        cur[k] = BatchRec{S, SF, P, D, (uint32_t)cnt, A, Bv, {0, 0, 0}};
        tl += (uint64_t)batch_size(k) * S + SF;
        nmet += cnt;
      }
      carry += (uint64_t)total;
    }
    wave_sync_lds();
    return Score{(int64_t)wave_sum_u64((uint64_t)nmet), wave_sum_u64(tl)};
  }

  // Leaving (o) and joining (e) request of changed batch k.
  __device__ __forceinline__ void out_in(int k, const Move &mv, int &o, int &e) const {
    int opos, epos;
    if (mv.type == 1) {  // swap
      const int lo = min(mv.i, mv.j), hi = max(mv.i, mv.j);
      opos = (k == mv.a) ? lo : hi;
      epos = (k == mv.a) ? hi : lo;
    } else if (mv.i < mv.j) {  // insert moving right: each batch passes its first member left
      opos = (k == mv.a) ? mv.i : k * B;
      epos = (k == mv.c) ? mv.i : (k + 1) * B;
    } else {  // insert moving left: each batch passes its last member right
      opos = (k == mv.c) ? mv.i : (k + 1) * B - 1;
      epos = (k == mv.a) ? mv.i : k * B - 1;
    }
    o = perm[opos];
    e = perm[epos];
  }

  // Batch-parallel pass over batches [k0, k1), all with unchanged members and starts
  // moved by `shift`: candidate records, their latency change, and a bitmask of the rows
  // holding a batch whose new start leaves its bounds (those need a member recount).
  __device__ uint64_t shift_range(int k0, int k1, int64_t shift, int64_t &dt_l) {
    uint64_t rows = 0;
    for (int kk0 = k0; kk0 < k1; kk0 += kWave) {
      const int kk = kk0 + lane;
      bool flip = false;
      if (kk < k1) {
        BatchRec b = cur[kk];
        b.S += (uint64_t)shift;
        flip = b.S > (uint64_t)b.A || b.S < (uint64_t)b.Bv;
        cand[kk] = b;
      }
      uint64_t f = __ballot(flip);
      while (f) {
        const int l = __builtin_ctzll(f);
        f &= f - 1;
        rows |= 1ull << ((kk0 + l) / G);
      }
    }
    if (lane == 0) dt_l += shift * requests_in(k0, k1);
    return rows;
  }

  // Candidate objective change of a move with a < c. Writes candidate F (speculative) and
  // candidate records for batches a..klast.
  __device__ void propose(const Move &mv, int64_t &dn, int64_t &dt, int &klast) {
    int64_t dn_l = 0, dt_l = 0;
    const int row_a = mv.a >> (6 - LG), row_c = mv.c >> (6 - LG);
    // rows holding changed batches: for a swap the rows of a and c, for an insert a..c
    int64_t carry = row_pass(row_a, mv, 0, true, dn_l, dt_l);
    const int64_t shift_mid = carry;  // start change of the batches between a and c (swap)
    uint64_t flagged = 0;
    if (mv.type == 2) {
      for (int row = row_a + 1; row <= row_c; ++row) carry += row_pass(row, mv, carry, true, dn_l, dt_l);
    } else if (row_c > row_a) {
      // the batches strictly between the two rows: their records are copied on accept, so
      // they are written even when the shift is 0 (no batch then leaves its bounds)
      if (row_c > row_a + 1) flagged |= shift_range((row_a + 1) * G, row_c * G, shift_mid, dt_l);
      carry += row_pass(row_c, mv, carry, true, dn_l, dt_l);
    }
    const int kb = (row_c + 1) * G;  // first batch after the rows of a..c
    if (carry != 0 && kb < M) {
      flagged |= shift_range(kb, M, carry, dt_l);
      klast = M - 1;
    } else {
      klast = min(kb - 1, M - 1);
    }
    // member-level recount of the rows holding a batch that left its bounds; their
    // latency change was already added by shift_range (sums of F are unchanged there)
    while (flagged) {
      const int row = __builtin_ctzll(flagged);
      flagged &= flagged - 1;
      row_pass(row, mv, row * G >= kb ? carry : shift_mid, false, dn_l, dt_l);
    }
    dn = Seg<LG>::leader_sum(dn_l);
    dt = Seg<LG>::leader_sum(dt_l);
  }

  // Restore F of the changed batches after a rejected proposal (reverse update).
  __device__ void undo(const Move &mv) {
    const int row_a = mv.a >> (6 - LG), row_c = mv.c >> (6 - LG);
    for (int row = row_a; row <= row_c; ++row) {
      if (mv.type == 1 && row != row_a && row != row_c) continue;
      const int k = row * G + seg;
      const int q = k * B + mm;
      const bool valid = mm < B && q < N;
      const bool seg_changed = k < M && mv.changes(k);
      int o = 0, e = 0;
      uint32_t Pold = 0;
      if (seg_changed) {
        out_in(k, mv, o, e);
        Pold = cur[k].P;
      }
      const Req ro = load_req(req, o), re = load_req(req, e);
      const uint32_t Pn = Pold + re.pf - ro.pf;
      int r = 0;
      Req rq{0, 0, 0, 0, 0};
      if (valid) {
        r = perm[q];
        rq = load_req(req, r);
      }
      const uint32_t to = (seg_changed && valid) ? w2(rq.L, rq.e, ro.L, sp.d2) : 0u;
      const uint32_t Fo = Pold + __umul24(ro.L, sp.d0) + (Seg<LG>::template all<OpAdd>(to, lane) >> 1);
      if (seg_changed && valid) {
        if (r == o) {
          F[o] = Fo;
        } else {
          const int32_t dw = (int32_t)(w2(ro.L, ro.e, rq.L, sp.d2) - w2(re.L, re.e, rq.L, sp.d2));
          F[r] = F[r] + (Pold - Pn) + (uint32_t)(dw >> 1);
        }
      }
    }
  }

  __device__ __forceinline__ void apply_move(int type, int i, int j) { apply_move_lds(perm, type, i, j, lane); }
};

// The request records of the static delta kernels, staged by the whole workgroup: n records
// and a zero spare record at index n.
__device__ __forceinline__ void load_static_records(const QueuePtrs &q, const DevModel &m, uint4 *req) {
  const int n = m.n;
  for (int r = threadIdx.x; r <= n; r += blockDim.x) {
    if (r == n) {
      req[r] = make_uint4(0u, 0u, 0u, 0u);  // spare record for lanes outside a batch
      continue;
    }
    const uint32_t lin = q.in_len[r], lout = q.out_len[r];
    const uint32_t pf = (uint32_t)(m.p0 + m.p1 * lin);
    const uint32_t e = (uint32_t)(2 * (m.d1 + m.d2 * lin) + m.d2);
    const uint32_t kind = q.kind[r];
    const uint64_t thr_l = (uint64_t)q.thr[r] * lout;
    const uint32_t thr = kind == 1 ? (uint32_t)min(thr_l, (uint64_t)0xFFFFFFFFu) : q.thr[r];
    req[r] = make_uint4(lin | (lout << 16), thr, kind | (e << 2), pf);
  }
}

// LDS of one chain of the row kernel: order, finish offsets, current and candidate batch records.
__host__ __device__ __forceinline__ size_t static_chain_bytes(int n, int B) {
  const size_t M = (size_t)(n + B - 1) / B;
  return (((size_t)n * 2 + 15) & ~size_t(15)) + (((size_t)(n + 1) * 4 + 15) & ~size_t(15)) + 2 * M * sizeof(BatchRec);
}

// One chain of the row kernel by one wave: record slot `chain`, Philox chain index
// `rng_chain`, the request records in `req`, the chain's LDS at `wb`.
template <int LG, int OBJ>
__device__ void anneal_static_body(const DevModel &m, const StaticParams &sp, const uint4 *req, unsigned char *wb,
                                   int chains, int chain, uint32_t rng_chain, int iters, double T0, double alpha,
                                   uint32_t key0, uint32_t key1, uint64_t swap_thr, const SearchParams &srch,
                                   unsigned char *ws) {
  const int n = m.n, B = m.B;
  const int M = (n + B - 1) / B;
  constexpr int G = kWave >> LG;
  const int R = (M + G - 1) / G;
  const size_t perm_b = ((size_t)n * 2 + 15) & ~size_t(15);
  const size_t f_b = ((size_t)(n + 1) * 4 + 15) & ~size_t(15);
  const size_t rec_b = (size_t)M * sizeof(BatchRec);
  const int lane = lane_id();
  StaticChain<LG> st{req,
                     reinterpret_cast<uint16_t *>(wb),
                     reinterpret_cast<uint32_t *>(wb + perm_b),
                     reinterpret_cast<BatchRec *>(wb + perm_b + f_b),
                     reinterpret_cast<BatchRec *>(wb + perm_b + f_b + rec_b),
                     sp, n, B, M, R, lane, lane >> LG, lane & ((1 << LG) - 1)};
  const WsHeader *h = reinterpret_cast<const WsHeader *>(ws);
  const int64_t t_ref = h->t_ref;
  const int64_t allmet = h->allmet;
  const uint16_t *start = reinterpret_cast<const uint16_t *>(ws + ws_off_start());
  const size_t stride = ws_perm_stride(n);
  uint16_t *gbest = reinterpret_cast<uint16_t *>(ws + ws_off_best(n, chains)) + (size_t)chain * stride;
  uint16_t *gcur = reinterpret_cast<uint16_t *>(ws + ws_off_cur(n, chains)) + (size_t)chain * stride;
  for (int p = lane; p < n; p += kWave) {
    const uint16_t v = start[p];
    st.perm[p] = v;
    gbest[p] = v;
  }
  wave_sync_lds();
  const Score s0 = st.init();
  int64_t cn = s0.n;
  uint64_t ct = s0.t;
  int64_t bn = cn;
  uint64_t bt = ct;
  int64_t biter = -1, accepts = 0;
  uint64_t digest = kFnvOffset;
  Cooling cool{T0, alpha, srch.level_len, srch.level_len};
  ProposalStream ps;
  const int iters_run = (srch.early_exit && allmet) ? 0 : iters;
  for (int k = 0; k < iters_run; ++k) {
    if ((k & (kWave - 1)) == 0) ps.refill(k, lane, n, rng_chain, key0, key1, swap_thr, 0);
    const uint32_t pk = ps.packed(k), w3 = ps.word3(k);
    const int i = (int)(pk & 1023u), j = (int)((pk >> 10) & 1023u);
    Move mv;
    mv.type = (int)((pk >> 20) & 1u) + 1;
    mv.i = i;
    mv.j = j;
    mv.a = (int)div_b((uint32_t)min(i, j), sp.bmagic);
    mv.c = (int)div_b((uint32_t)max(i, j), sp.bmagic);
    bool acc;
    if (mv.a == mv.c) {
      // same batch: every batch keeps its members, the objective is unchanged
      acc = true;
      st.apply_move(mv.type, i, j);
    } else {
      int64_t dn, dt;
      int klast;
      st.propose(mv, dn, dt, klast);
      acc = obj_accept<OBJ>(cn, ct, dn, dt, t_ref, cool.T, w3);
      if (acc) {
        st.apply_move(mv.type, i, j);
        for (int kk = mv.a + lane; kk <= klast; kk += kWave) st.cur[kk] = st.cand[kk];
        wave_sync_lds();
        cn += dn;
        ct += (uint64_t)dt;
      } else {
        st.undo(mv);
        wave_sync_lds();
      }
    }
    if (acc) {
      ++accepts;
      digest = (digest ^ (uint64_t)k) * kFnvPrime;
      digest = (digest ^ (uint64_t)cn) * kFnvPrime;
      digest = (digest ^ ct) * kFnvPrime;
      if (obj_better<OBJ>(cn, ct, bn, bt)) {
        bn = cn;
        bt = ct;
        biter = k;
        for (int p = lane; p < n; p += kWave) gbest[p] = st.perm[p];
      }
    }
    cool.step();
  }
  for (int p = lane; p < n; p += kWave) gcur[p] = st.perm[p];
  if (lane == 0) {
    int64_t *rec = reinterpret_cast<int64_t *>(ws + ws_off_records(n)) + (size_t)chain * 8;
    rec[0] = cn;
    rec[1] = (int64_t)ct;
    rec[2] = bn;
    rec[3] = (int64_t)bt;
    rec[4] = biter;
    rec[5] = accepts;
    rec[6] = (int64_t)digest;
    rec[7] = allmet;
  }
}

// One wave per chain; blockDim / 64 chains per workgroup.
template <int LG, int OBJ>
__global__ void __launch_bounds__(1024) anneal_static_kernel(DevModel m, StaticParams sp, QueuePtrs q, int chains,
                                                              int iters, double T0, double alpha, uint32_t key0,
                                                              uint32_t key1, uint64_t swap_thr, SearchParams srch,
                                                              unsigned char *ws) {
  extern __shared__ __align__(16) unsigned char lds[];
  if (!gate_open(ws, m.gate, m.flags)) return;
  const int n = m.n;
  const int waves = blockDim.x >> 6;
  uint4 *req = reinterpret_cast<uint4 *>(lds);
  const int wave = uniform((int)(threadIdx.x >> 6));
  unsigned char *wb = lds + (size_t)(n + 1) * 16 + (size_t)wave * static_chain_bytes(n, m.B);
  load_static_records(q, m, req);
  __syncthreads();
  const int chain = uniform((int)blockIdx.x * waves + wave);
  if (chain >= chains) return;
  anneal_static_body<LG, OBJ>(m, sp, req, wb, chains, chain, (uint32_t)chain, iters, T0, alpha, key0, key1, swap_thr,
                              srch, ws);
}

}  // namespace sa

namespace sa {

// Evaluation of whole orders under static admission, one wave per order, with the same
// 32-bit arithmetic as the annealing kernel: per batch the prefill sum, each member's
// finish offset by the pairwise closed form (one 8-byte LDS read and three 24-bit ops
// per pair), the batch duration, the start scan across batches and the SLO test.
// T32: every time on the timeline fits 32 bits (the host's check; not with DETAIL): the batch
// starts come from a 32-bit scan of the batch durations that begins at the batch size (the
// duration is the same on every lane of a batch) and the latency sum from 16-bit halves.
template <int LG, bool DETAIL, bool T32 = false>
__global__ void __launch_bounds__(256) eval_static_kernel(DevModel m, StaticParams sp, QueuePtrs q,
                                                           const uint16_t *__restrict__ perms, int64_t rows,
                                                           int64_t *__restrict__ out, int64_t *__restrict__ detail) {
  extern __shared__ __align__(16) unsigned char lds[];
  const EvalRows span = eval_gate(q, m, rows, out);
  if (span.end <= span.begin) return;
  constexpr int Bp = 1 << LG, G = kWave >> LG;
  const int n = m.n, B = m.B;
  const int M = (n + B - 1) / B, R = (M + G - 1) / G;
  uint4 *req = reinterpret_cast<uint4 *>(lds);
  const size_t perm_b = ((size_t)n * 2 + 15) & ~size_t(15);
  const size_t per_wave = perm_b + 64 * 8 + 32 * 4;
  const int wave = uniform((int)(threadIdx.x >> 6));
  const int waves = blockDim.x >> 6;
  unsigned char *wb = lds + (size_t)(n + 1) * 16 + (size_t)wave * per_wave;
  uint16_t *perm = reinterpret_cast<uint16_t *>(wb);
  uint2 *stage = reinterpret_cast<uint2 *>(wb + perm_b);
  uint32_t *bitmap = reinterpret_cast<uint32_t *>(wb + perm_b + 64 * 8);
  for (int r = threadIdx.x; r <= n; r += blockDim.x) {
    if (r == n) {
      req[r] = make_uint4(0u, 0u, 0u, 0u);
      continue;
    }
    const uint32_t lin = q.in_len[r], lout = q.out_len[r];
    const uint32_t pf = (uint32_t)(m.p0 + m.p1 * lin);
    const uint32_t e = (uint32_t)(2 * (m.d1 + m.d2 * lin) + m.d2);
    const uint32_t kind = q.kind[r];
    const uint64_t thr_l = (uint64_t)q.thr[r] * lout;
    const uint32_t thr = kind == 1 ? (uint32_t)min(thr_l, (uint64_t)0xFFFFFFFFu) : q.thr[r];
    req[r] = make_uint4(lin | (lout << 16), thr, kind | (e << 2), pf);
  }
  __syncthreads();
  const int lane = lane_id();
  const int seg = lane >> LG, mm = lane & (Bp - 1);
  const uint32_t d2m = sp.d2 & 0xFFFFFFu;
  for (int64_t row = span.begin + (int64_t)blockIdx.x * waves + wave; row < span.end;
       row += (int64_t)gridDim.x * waves) {
    const uint16_t *src = perms + row * n;
    if (lane < 32) bitmap[lane] = 0u;
    wave_sync_lds();
    bool bad = false;
    for (int p = lane; p < n; p += kWave) {
      const uint32_t v = src[p];
      perm[p] = (uint16_t)v;
      if (v >= (uint32_t)n) {
        bad = true;
      } else {
        const uint32_t bit = 1u << (v & 31u);
        if (atomicOr(&bitmap[v >> 5], bit) & bit) bad = true;
      }
    }
    wave_sync_lds();
    if (__ballot(bad) != 0ull) {
      if (lane == 0) {
        out[2 * row] = -1;
        out[2 * row + 1] = -1;
      }
      continue;
    }
    uint64_t carry = 0, tl = 0;
    uint32_t carry32 = 0, tlo = 0, thi = 0;
    int nmet = 0;
    for (int rr = 0; rr < R; ++rr) {
      const int k = rr * G + seg;
      const int qpos = k * B + mm;
      const bool valid = mm < B && qpos < n;
      const int r = valid ? (int)perm[min(qpos, n - 1)] : n;
      const Req x = load_req(req, r);
      stage[lane] = make_uint2(x.L, x.e);
      wave_sync_lds();
      const uint32_t P = Seg<LG>::template all<OpAdd>(x.pf, lane);
      uint32_t acc = 0;
      const int base = seg << LG;
      // 24-bit products: d2 mu + e_j < 2^24 and mu (d2 mu + e_j) < 2^32 (host width check);
      // four members per step so that their reads go out together
      auto pair = [&](const uint2 sj) {
        const uint32_t mu = min(sj.x, x.L);
        acc = mad24_v(mu, mad24_v(d2m, mu, sj.y), acc);
      };
      int jj = 0;
      for (; jj + 4 <= B; jj += 4) {
        const uint2 s0 = stage[base + jj], s1 = stage[base + jj + 1], s2 = stage[base + jj + 2],
                    s3 = stage[base + jj + 3];
        pair(s0);
        pair(s1);
        pair(s2);
        pair(s3);
      }
      for (; jj < B; ++jj) pair(stage[base + jj]);
      wave_sync_lds();
      const uint32_t F = valid ? P + __umul24(x.L, sp.d0) + (acc >> 1) : 0u;
      const uint32_t D = Seg<LG>::template all<OpMax>(F, lane);
      const Slack sl = slack_of(x.kind, x.thr, x.L, P, F);
      if constexpr (T32) {
        // inclusive sum of the durations of the round's batches up to the lane's (lanes past
        // the last batch hold D = 0)
        uint32_t v = D;
        if constexpr (LG <= 0) v += dpp_old<kDppRowShr1, 0xF>(0u, v);
        if constexpr (LG <= 1) v += dpp_old<kDppRowShr2, 0xF>(0u, v);
        if constexpr (LG <= 2) v += dpp_old<kDppRowShr4, 0xF>(0u, v);
        if constexpr (LG <= 3) v += dpp_old<kDppRowShr8, 0xF>(0u, v);
        if constexpr (LG <= 4) v += dpp_old<kDppRowBcast15, 0xA>(0u, v);
        if constexpr (LG <= 5) v += dpp_old<kDppRowBcast31, 0xC>(0u, v);
        const uint32_t S = carry32 + v - D;
        const bool met = valid && slack_met(sl, S);
        nmet += __popcll(__ballot(met));
        const uint32_t e2e = S + F;
        tlo += valid ? (e2e & 0xFFFFu) : 0u;
        thi += valid ? (e2e >> 16) : 0u;
        carry32 += readlane(v, kWave - 1);
      } else {
        int64_t excl, total;
        Seg<LG>::scan(k < M ? (int64_t)D : 0, lane, excl, total);
        const uint64_t S = carry + (uint64_t)excl;
        const bool met = valid && slack_met(sl, S);
        nmet += __popcll(__ballot(met));
        if (valid) {
          tl += S + F;
          if (DETAIL) {
            detail[row * n * 2 + 2 * r] = (int64_t)(S + P);
            detail[row * n * 2 + 2 * r + 1] = (int64_t)(S + F);
          }
        }
        carry += (uint64_t)total;
      }
    }
    uint64_t t;
    if constexpr (T32) {
      // each lane's halves below 2^20 (at most 16 rounds), their wave sums below 2^26
      Seg<6>::template all2<OpAdd, OpAdd>(tlo, thi, lane);
      t = (uint64_t)tlo + ((uint64_t)thi << 16);
    } else {
      t = wave_sum_u64(tl);
    }
    if (lane == 0) {
      out[2 * row] = nmet;
      out[2 * row + 1] = (int64_t)t;
    }
    wave_sync_lds();
  }
}

}  // namespace sa
