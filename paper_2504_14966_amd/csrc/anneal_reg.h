// Annealing chains under static admission for small queues, state in registers (gfx950).
//
// For at most 64 requests and a batch size of 1, 2, 4, 8 or 16, lane p holds the request at
// position p of the order: its output length and id, its pair-cost parameter e = 2 (d1 + d2
// l_in) + d2 and kind, its prefill and its SLO threshold (for TPOT, threshold times output
// length, saturated at 2^32 - 1). Batch k is lanes [kB, kB + B), inside one DPP row. A
// proposal builds the candidate order in registers (a swap is two v_readlane and two
// v_writelane per field; an insert is one DPP wave shift, a range select and one
// v_writelane) and replays it in full with no LDS traffic:
//   - each member's finish offset F = P + L d0 + (sum over the batch's members j of
//     mu (e_j + d2 mu)) / 2, mu = min(L_j, L), the batch's members reached by rotating the
//     row (row_ror, or the two rotations that stay inside an 8-lane half, or quad
//     permutations); the rotations read the same source registers, so they are independent;
//   - the batch prefill P and duration D by segment all-reduces, the batch starts by an
//     exclusive add-scan of D (32-bit, starting at the batch size, when the device check
//     bounds the whole timeline below 2^32; else 64-bit from each batch's last lane);
//   - TTFT = S + P, e2e = S + F and the SLO tests per lane; the met count by ballot, the
//     latency sum by two 32-bit reductions of 16-bit halves (or one 64-bit reduction).
// A move inside one batch changes no member's times and needs no replay. The 32-bit
// products and sums are exact under the fixed-size delta kernel's width checks.
#pragma once
#include "anneal_sized.h"
#include "anneal_wave.h"
#include "fit.h"

namespace sa {

// The small-queue kernel's applicability: n <= 64 and B a power of two up to 16.
__host__ __device__ __forceinline__ bool reg_kernel_fits(int n, int B) {
  return n >= 1 && n <= 64 && B >= 1 && B <= 16 && (B & (B - 1)) == 0;
}

template <int CTRL>
__device__ __forceinline__ uint32_t dppv(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, true);
}

// sum over the other members j of the lane's batch of mu (e_j + d2 mu), mu = min(L_j, L)
template <int LG>
__device__ __forceinline__ uint32_t pair_sum_others(uint32_t L, uint32_t e, uint32_t d2, int lane) {
  uint32_t acc = 0;
  auto term = [&](uint32_t Lj, uint32_t ej) {
    const uint32_t mu = min(Lj, L);
    acc = mad24_v(mu, mad24_v(d2, mu, ej), acc);
  };
  if constexpr (LG == 1) {
    term(dppv<0xB1>(L), dppv<0xB1>(e));  // quad_perm [1,0,3,2]
  } else if constexpr (LG == 2) {
    term(dppv<0x39>(L), dppv<0x39>(e));  // quad_perm [1,2,3,0]
    term(dppv<0x4E>(L), dppv<0x4E>(e));  // quad_perm [2,3,0,1]
    term(dppv<0x93>(L), dppv<0x93>(e));  // quad_perm [3,0,1,2]
  } else if constexpr (LG == 3) {
    // rotate by r inside the lane's 8-lane half: row_ror:r where that stays in the half,
    // else row_ror:(r + 8)
    const int m8 = lane & 7;
#pragma unroll
    for (int r = 1; r < 8; ++r) {
      uint32_t La, ea, Lb, eb;
      switch (r) {
        case 1: La = dppv<0x121>(L); ea = dppv<0x121>(e); Lb = dppv<0x129>(L); eb = dppv<0x129>(e); break;
        case 2: La = dppv<0x122>(L); ea = dppv<0x122>(e); Lb = dppv<0x12A>(L); eb = dppv<0x12A>(e); break;
        case 3: La = dppv<0x123>(L); ea = dppv<0x123>(e); Lb = dppv<0x12B>(L); eb = dppv<0x12B>(e); break;
        case 4: La = dppv<0x124>(L); ea = dppv<0x124>(e); Lb = dppv<0x12C>(L); eb = dppv<0x12C>(e); break;
        case 5: La = dppv<0x125>(L); ea = dppv<0x125>(e); Lb = dppv<0x12D>(L); eb = dppv<0x12D>(e); break;
        case 6: La = dppv<0x126>(L); ea = dppv<0x126>(e); Lb = dppv<0x12E>(L); eb = dppv<0x12E>(e); break;
        default: La = dppv<0x127>(L); ea = dppv<0x127>(e); Lb = dppv<0x12F>(L); eb = dppv<0x12F>(e); break;
      }
      const bool same = m8 >= r;  // lane - r stays inside the half
      term(same ? La : Lb, same ? ea : eb);
    }
  } else if constexpr (LG == 4) {
#define SA_ROR(R) term(dppv<0x120 + (R)>(L), dppv<0x120 + (R)>(e));
    SA_ROR(1) SA_ROR(2) SA_ROR(3) SA_ROR(4) SA_ROR(5) SA_ROR(6) SA_ROR(7) SA_ROR(8)
    SA_ROR(9) SA_ROR(10) SA_ROR(11) SA_ROR(12) SA_ROR(13) SA_ROR(14) SA_ROR(15)
#undef SA_ROR
  }
  return acc;
}

// A move on positions held one per lane, as the byte address of each lane's source lane:
// a swap exchanges lanes i and `to`; an insert moves lane i to lane `to` and shifts the lanes
// between by one toward i. Every field of the candidate is then one lane permute
// (ds_bpermute) with this address, instead of v_readlane / v_writelane pairs whose scalar
// hand-offs serialise.
__device__ __forceinline__ int move_src_addr(bool swap, int i, int to, int lane) {
  int src;
  if (swap) {
    src = lane == i ? to : (lane == to ? i : lane);
  } else {
    const bool right = i < to;
    const int lo = right ? i : to + 1;
    const uint32_t span = (uint32_t)(right ? to - i : i - to);
    src = lane == to ? i : ((uint32_t)(lane - lo) < span ? lane + (right ? 1 : -1) : lane);
  }
  return src << 2;
}
__device__ __forceinline__ uint32_t from_lane(int addr, uint32_t x) {
  return (uint32_t)__builtin_amdgcn_ds_bpermute(addr, (int)x);
}

// 64-bit all-reduce (sum) over the wave, result in every lane
__device__ __forceinline__ uint64_t wave_sum64_dpp(uint64_t v) {
  const uint64_t incl = scan_add64(v);
  return rl64(incl, kWave - 1);
}

struct RegState {
  uint32_t A;  // output length | request id << 16
  uint32_t E;  // e | kind << 30
  uint32_t PF, T;
};

// Full replay of the order held in registers: (met count, total latency). T32: every time on
// the timeline of any order fits 32 bits (the host's check), so the batch starts and the
// latency sum run in 32-bit lanes.
template <int LG, bool T32>
__device__ __forceinline__ Score reg_replay(const RegState &s, int n, uint32_t d0, uint32_t d2, int lane) {
  constexpr int B = 1 << LG;
  const bool valid = lane < n;
  const uint32_t L = s.A & 0xFFFFu, e = s.E & 0x3FFFFFFFu, kind = s.E >> 30;
  const uint32_t acc = mad24_v(L, mad24_v(d2, L, e), pair_sum_others<LG>(L, e, d2, lane));
  const uint32_t P = Seg<LG>::template all<OpAdd>(s.PF, lane);
  const uint32_t F = valid ? P + __umul24(L, d0) + (acc >> 1) : 0u;
  const uint32_t D = Seg<LG>::template all<OpMax>(F, lane);
  if constexpr (T32) {
    // inclusive sum of the batch durations up to the lane's batch: D is the same on every
    // lane of a batch, so the in-row shifts start at the batch size
    uint32_t v = D;
    if constexpr (LG <= 0) v += dpp_old<kDppRowShr1, 0xF>(0u, v);
    if constexpr (LG <= 1) v += dpp_old<kDppRowShr2, 0xF>(0u, v);
    if constexpr (LG <= 2) v += dpp_old<kDppRowShr4, 0xF>(0u, v);
    if constexpr (LG <= 3) v += dpp_old<kDppRowShr8, 0xF>(0u, v);
    v += dpp_old<kDppRowBcast15, 0xA>(0u, v);
    v += dpp_old<kDppRowBcast31, 0xC>(0u, v);
    const uint32_t S = v - D;
    const uint32_t ttft = S + P, e2e = S + F;
    const uint32_t x = kind == 0 ? ttft : (kind == 2 ? e2e : F - P);
    const int64_t nmet = __popcll(__ballot(valid && x <= s.T));
    // the latency sum: 16-bit halves of the 32-bit latencies, each sum below 2^22
    uint32_t lo = valid ? (e2e & 0xFFFFu) : 0u, hi = valid ? (e2e >> 16) : 0u;
    wave_all2<OpAdd, OpAdd>(lo, hi);
    return Score{nmet, (uint64_t)lo + ((uint64_t)hi << 16)};
  } else {
    const uint64_t contrib = (lane & (B - 1)) == B - 1 ? (uint64_t)D : 0ull;
    const uint64_t S = scan_add64(contrib) - contrib;
    const uint64_t ttft = S + P, e2e = S + F;
    const bool met = valid && (kind == 0 ? ttft <= (uint64_t)s.T : (kind == 2 ? e2e <= (uint64_t)s.T : F - P <= s.T));
    const int64_t nmet = __popcll(__ballot(met));
    return Score{nmet, wave_sum64_dpp(valid ? e2e : 0ull)};
  }
}

// One chain by one wave: record slot `chain`, Philox chain index `rng_chain`.
template <int LG, int OBJ, bool T32>
__device__ void anneal_reg_body(const DevModel &m, const QueuePtrs &q, int chains, int chain, uint32_t rng_chain,
                                int iters, double T0, double alpha, uint32_t key0, uint32_t key1, uint64_t swap_thr,
                                const SearchParams &srch, unsigned char *ws) {
  const int n = m.n;
  const int lane = lane_id();
  const uint32_t d0 = (uint32_t)m.d0, d2 = (uint32_t)m.d2;
  const WsHeader *h = reinterpret_cast<const WsHeader *>(ws);
  const int64_t t_ref = h->t_ref;
  const int64_t allmet = h->allmet;
  const uint16_t *start = reinterpret_cast<const uint16_t *>(ws + ws_off_start());
  const size_t stride = ws_perm_stride(n);
  uint16_t *gbest = reinterpret_cast<uint16_t *>(ws + ws_off_best(n, chains)) + (size_t)chain * stride;
  uint16_t *gcur = reinterpret_cast<uint16_t *>(ws + ws_off_cur(n, chains)) + (size_t)chain * stride;
  RegState cur{0u, 0u, 0u, 0u};
  if (lane < n) {
    const uint32_t r = start[lane];
    const uint32_t lin = q.in_len[r], L = q.out_len[r], kind = q.kind[r], thr = q.thr[r];
    const uint32_t e = (uint32_t)(2 * (m.d1 + m.d2 * lin) + m.d2);
    const uint64_t thr_l = (uint64_t)thr * L;
    cur.A = L | (r << 16);
    cur.E = e | (kind << 30);
    cur.PF = (uint32_t)(m.p0 + m.p1 * lin);
    cur.T = kind == 1 ? (uint32_t)min(thr_l, (uint64_t)0xFFFFFFFFu) : thr;
    gbest[lane] = (uint16_t)r;
  }
  const Score s0 = reg_replay<LG, T32>(cur, n, d0, d2, lane);
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
    // swap positions i and j, or insert the request at i at j (the ones between shift by
    // one toward i)
    const int addr = move_src_addr(((pk >> 20) & 1u) == 0u, i, j, lane);
    const RegState cand{from_lane(addr, cur.A), from_lane(addr, cur.E), from_lane(addr, cur.PF), from_lane(addr, cur.T)};
    // a move inside one batch keeps every batch's members: the score is unchanged (and the
    // move is kept under either objective), so the replay is skipped
    const Score s = (i >> LG) == (j >> LG) ? Score{cn, ct} : reg_replay<LG, T32>(cand, n, d0, d2, lane);
    const bool acc = obj_accept<OBJ>(cn, ct, s.n - cn, (int64_t)(s.t - ct), t_ref, cool.T, w3);
    if (acc) {
      cur = cand;
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
        if (lane < n) gbest[lane] = (uint16_t)(cur.A >> 16);
      }
    }
    cool.step();
  }
  if (lane < n) gcur[lane] = (uint16_t)(cur.A >> 16);
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

// One wave per chain; blockDim / 64 chains per workgroup; no LDS.
template <int LG, int OBJ>
__global__ void __launch_bounds__(256) anneal_reg_kernel(DevModel m, QueuePtrs q, int chains, int iters, double T0,
                                                          double alpha, uint32_t key0, uint32_t key1,
                                                          uint64_t swap_thr, SearchParams srch, unsigned char *ws) {
  if (!gate_open(ws, m.gate, m.flags)) return;
  const int waves = blockDim.x >> 6;
  const int chain = uniform((int)blockIdx.x * waves + (int)(threadIdx.x >> 6));
  if (chain >= chains) return;
  if (m.flags & kFlagTime32)
    anneal_reg_body<LG, OBJ, true>(m, q, chains, chain, (uint32_t)chain, iters, T0, alpha, key0, key1, swap_thr, srch,
                                   ws);
  else
    anneal_reg_body<LG, OBJ, false>(m, q, chains, chain, (uint32_t)chain, iters, T0, alpha, key0, key1, swap_thr, srch,
                                    ws);
}

// ---- 65 to 192 requests: H = 2 or 3 positions per lane ----
//
// Position p sits in lane p mod 64 of part p / 64 (H registers per field). Batches of at
// most 16 never straddle the parts, so each part replays as above; a part's batch starts
// add the earlier parts' totals. A swap reads and writes the two positions in their parts;
// an insert shifts each part by one DPP wave shift and carries the element that crosses a
// part boundary with one v_readlane and one v_writelane.

__host__ __device__ __forceinline__ int reg_parts(int n, int B) {
  if (n < 1 || n > 192 || B < 1 || B > 16 || (B & (B - 1)) != 0) return 0;
  return (n + 63) / 64;
}

template <int H>
struct RegStateH {
  RegState h[H];
};

// lane l of x[part] for a wave-uniform part index (scalar branches around each v_readlane,
// so that no dynamically indexed register array is formed)
template <int H>
__device__ __forceinline__ uint32_t read_part(const uint32_t (&x)[H], int part, int l) {
  if (H > 2 && part == 2) return readlane(x[H > 2 ? 2 : 0], l);
  if (part == 1) return readlane(x[1], l);
  return readlane(x[0], l);
}

// A part's own values: each member's finish offset F within its batch, and its batch's
// prefill P and duration D (the same on every lane of a batch).
struct PartVals {
  uint32_t F, P, D;
};

template <int LG>
__device__ __forceinline__ PartVals part_local(const RegState &st, bool valid, uint32_t d0, uint32_t d2, int lane) {
  const uint32_t L = st.A & 0xFFFFu, e = st.E & 0x3FFFFFFFu;
  const uint32_t acc = mad24_v(L, mad24_v(d2, L, e), pair_sum_others<LG>(L, e, d2, lane));
  const uint32_t P = Seg<LG>::template all<OpAdd>(st.PF, lane);
  const uint32_t F = valid ? P + __umul24(L, d0) + (acc >> 1) : 0u;
  return PartVals{F, P, Seg<LG>::template all<OpMax>(F, lane)};
}

// Starts across the parts, SLO tests and sums from the parts' values.
template <int LG, bool T32, int H>
__device__ __forceinline__ Score part_combine(const RegStateH<H> &s, const PartVals (&pv)[H], int n, int lane) {
  constexpr int B = 1 << LG;
  int64_t nmet = 0;
  if constexpr (T32) {
    uint32_t lo = 0, hi = 0, carry = 0;
#pragma unroll
    for (int h = 0; h < H; ++h) {
      const bool valid = lane + 64 * h < n;
      const uint32_t kind = s.h[h].E >> 30, D = pv[h].D, F = pv[h].F, P = pv[h].P;
      uint32_t v = D;
      if constexpr (LG <= 0) v += dpp_old<kDppRowShr1, 0xF>(0u, v);
      if constexpr (LG <= 1) v += dpp_old<kDppRowShr2, 0xF>(0u, v);
      if constexpr (LG <= 2) v += dpp_old<kDppRowShr4, 0xF>(0u, v);
      if constexpr (LG <= 3) v += dpp_old<kDppRowShr8, 0xF>(0u, v);
      v += dpp_old<kDppRowBcast15, 0xA>(0u, v);
      v += dpp_old<kDppRowBcast31, 0xC>(0u, v);
      const uint32_t S = carry + v - D;
      const uint32_t ttft = S + P, e2e = S + F;
      const uint32_t x = kind == 0 ? ttft : (kind == 2 ? e2e : F - P);
      nmet += __popcll(__ballot(valid && x <= s.h[h].T));
      lo += valid ? (e2e & 0xFFFFu) : 0u;
      hi += valid ? (e2e >> 16) : 0u;
      carry += readlane(v, kWave - 1);
    }
    // each lane's halves below 2^18, their sums below 2^24
    wave_all2<OpAdd, OpAdd>(lo, hi);
    return Score{nmet, (uint64_t)lo + ((uint64_t)hi << 16)};
  } else {
    uint64_t carry = 0, tsum = 0;
#pragma unroll
    for (int h = 0; h < H; ++h) {
      const bool valid = lane + 64 * h < n;
      const uint32_t kind = s.h[h].E >> 30, F = pv[h].F, P = pv[h].P;
      const uint64_t contrib = (lane & (B - 1)) == B - 1 ? (uint64_t)pv[h].D : 0ull;
      const uint64_t incl = scan_add64(contrib);
      const uint64_t S = carry + incl - contrib;
      const uint64_t ttft = S + P, e2e = S + F;
      const bool met = valid && (kind == 0   ? ttft <= (uint64_t)s.h[h].T
                                 : kind == 2 ? e2e <= (uint64_t)s.h[h].T
                                             : F - P <= s.h[h].T);
      nmet += __popcll(__ballot(met));
      tsum += valid ? e2e : 0ull;
      carry += rl64(incl, kWave - 1);
    }
    return Score{nmet, wave_sum64_dpp(tsum)};
  }
}

template <int LG, int OBJ, bool T32, int H>
__device__ void anneal_reg_h_body(const DevModel &m, const QueuePtrs &q, int chains, int chain, uint32_t rng_chain,
                                  int iters, double T0, double alpha, uint32_t key0, uint32_t key1, uint64_t swap_thr,
                                  const SearchParams &srch, unsigned char *ws) {
  const int n = m.n;
  const int lane = lane_id();
  const uint32_t d0 = (uint32_t)m.d0, d2 = (uint32_t)m.d2;
  const WsHeader *hd = reinterpret_cast<const WsHeader *>(ws);
  const int64_t t_ref = hd->t_ref;
  const int64_t allmet = hd->allmet;
  const uint16_t *start = reinterpret_cast<const uint16_t *>(ws + ws_off_start());
  const size_t stride = ws_perm_stride(n);
  uint16_t *gbest = reinterpret_cast<uint16_t *>(ws + ws_off_best(n, chains)) + (size_t)chain * stride;
  uint16_t *gcur = reinterpret_cast<uint16_t *>(ws + ws_off_cur(n, chains)) + (size_t)chain * stride;
  RegStateH<H> cur;
#pragma unroll
  for (int h = 0; h < H; ++h) {
    cur.h[h] = RegState{0u, 0u, 0u, 0u};
    const int p = lane + 64 * h;
    if (p < n) {
      const uint32_t r = start[p];
      const uint32_t lin = q.in_len[r], L = q.out_len[r], kind = q.kind[r], thr = q.thr[r];
      const uint32_t e = (uint32_t)(2 * (m.d1 + m.d2 * lin) + m.d2);
      const uint64_t thr_l = (uint64_t)thr * L;
      cur.h[h].A = L | (r << 16);
      cur.h[h].E = e | (kind << 30);
      cur.h[h].PF = (uint32_t)(m.p0 + m.p1 * lin);
      cur.h[h].T = kind == 1 ? (uint32_t)min(thr_l, (uint64_t)0xFFFFFFFFu) : thr;
      gbest[p] = (uint16_t)r;
    }
  }
  // each part's values are kept with the state; a proposal recomputes only the parts that
  // hold a changed position (the finish offsets move with their requests in the others)
  PartVals cpv[H];
#pragma unroll
  for (int h = 0; h < H; ++h) cpv[h] = part_local<LG>(cur.h[h], lane + 64 * h < n, d0, d2, lane);
  const Score s0 = part_combine<LG, T32, H>(cur, cpv, n, lane);
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
    const int pi = i >> 6, li = i & 63, pj = j >> 6, lj = j & 63;
    const bool swap = ((pk >> 20) & 1u) == 0u;
    RegStateH<H> cand;
    PartVals npv[H];
    // one per-position field across the parts (x in, y out)
    auto move = [&](const uint32_t (&x)[H], uint32_t (&y)[H]) {
      const uint32_t xi = read_part<H>(x, pi, li);
      if (swap) {
        const uint32_t xj = read_part<H>(x, pj, lj);
#pragma unroll
        for (int h = 0; h < H; ++h) {
          y[h] = x[h];
          if (h == pi) y[h] = wlane_m0(xj, li, y[h]);
          if (h == pj) y[h] = wlane_m0(xi, lj, y[h]);
        }
      } else {
        // insert: the request at i moves to j; positions [i, j) take p + 1, or (j, i] take
        // p - 1
        const bool right = i < j;
        const int lo = right ? i : j + 1;
        const uint32_t span = (uint32_t)(right ? j - i : i - j);
#pragma unroll
        for (int h = 0; h < H; ++h) {
          uint32_t sh;
          if (right) {
            sh = dppv<0x130>(x[h]);
            if (h + 1 < H) sh = wlane_m0(readlane(x[h + 1 < H ? h + 1 : h], 0), kWave - 1, sh);
          } else {
            sh = dppv<0x138>(x[h]);
            if (h > 0) sh = wlane_m0(readlane(x[h > 0 ? h - 1 : 0], kWave - 1), 0, sh);
          }
          y[h] = (uint32_t)(lane + 64 * h - lo) < span ? sh : x[h];
          if (h == pj) y[h] = wlane_m0(xi, lj, y[h]);
        }
      }
    };
    {
      uint32_t x[H], y[H];
#define SA_MOVE_FIELD(GET, PUT)                      \
  _Pragma("unroll") for (int h = 0; h < H; ++h) x[h] = GET; \
  move(x, y);                                        \
  _Pragma("unroll") for (int h = 0; h < H; ++h) PUT = y[h];
      SA_MOVE_FIELD(cur.h[h].A, cand.h[h].A)
      SA_MOVE_FIELD(cur.h[h].E, cand.h[h].E)
      SA_MOVE_FIELD(cur.h[h].PF, cand.h[h].PF)
      SA_MOVE_FIELD(cur.h[h].T, cand.h[h].T)
      SA_MOVE_FIELD(cpv[h].F, npv[h].F)
#undef SA_MOVE_FIELD
    }
#pragma unroll
    for (int h = 0; h < H; ++h) {
      npv[h].P = cpv[h].P;
      npv[h].D = cpv[h].D;
    }
    Score sc{cn, ct};
    // a move inside one batch keeps every batch's members and every member's offset: no
    // replay (the offsets moved with their requests)
    if ((i >> LG) != (j >> LG)) {
      const int plo = min(pi, pj), phi = max(pi, pj);
#pragma unroll
      for (int h = 0; h < H; ++h) {
        const bool touched = swap ? (h == pi || h == pj) : (h >= plo && h <= phi);
        if (touched) npv[h] = part_local<LG>(cand.h[h], lane + 64 * h < n, d0, d2, lane);
      }
      sc = part_combine<LG, T32, H>(cand, npv, n, lane);
    }
    if (obj_accept<OBJ>(cn, ct, sc.n - cn, (int64_t)(sc.t - ct), t_ref, cool.T, w3)) {
      cur = cand;
#pragma unroll
      for (int h = 0; h < H; ++h) cpv[h] = npv[h];
      cn = sc.n;
      ct = sc.t;
      ++accepts;
      digest = (digest ^ (uint64_t)k) * kFnvPrime;
      digest = (digest ^ (uint64_t)cn) * kFnvPrime;
      digest = (digest ^ ct) * kFnvPrime;
      if (obj_better<OBJ>(cn, ct, bn, bt)) {
        bn = cn;
        bt = ct;
        biter = k;
#pragma unroll
        for (int h = 0; h < H; ++h)
          if (lane + 64 * h < n) gbest[lane + 64 * h] = (uint16_t)(cur.h[h].A >> 16);
      }
    }
    cool.step();
  }
#pragma unroll
  for (int h = 0; h < H; ++h)
    if (lane + 64 * h < n) gcur[lane + 64 * h] = (uint16_t)(cur.h[h].A >> 16);
  if (lane == 0) write_record(ws, n, chain, cn, ct, bn, bt, biter, accepts, digest, allmet);
}

// The chain body for any request count the register kernels take (at most 192): one, two
// or three positions per lane.
template <int LG, int OBJ>
__device__ __forceinline__ void anneal_reg_any(const DevModel &m, const QueuePtrs &q, int chains, int chain,
                                               uint32_t rng_chain, int iters, double T0, double alpha, uint32_t key0,
                                               uint32_t key1, uint64_t swap_thr, const SearchParams &srch,
                                               unsigned char *ws) {
  const bool t32 = (m.flags & kFlagTime32) != 0;
  if (m.n <= 64) {
    if (t32) anneal_reg_body<LG, OBJ, true>(m, q, chains, chain, rng_chain, iters, T0, alpha, key0, key1, swap_thr, srch, ws);
    else anneal_reg_body<LG, OBJ, false>(m, q, chains, chain, rng_chain, iters, T0, alpha, key0, key1, swap_thr, srch, ws);
  } else if (m.n <= 128) {
    if (t32) anneal_reg_h_body<LG, OBJ, true, 2>(m, q, chains, chain, rng_chain, iters, T0, alpha, key0, key1, swap_thr, srch, ws);
    else anneal_reg_h_body<LG, OBJ, false, 2>(m, q, chains, chain, rng_chain, iters, T0, alpha, key0, key1, swap_thr, srch, ws);
  } else {
    if (t32) anneal_reg_h_body<LG, OBJ, true, 3>(m, q, chains, chain, rng_chain, iters, T0, alpha, key0, key1, swap_thr, srch, ws);
    else anneal_reg_h_body<LG, OBJ, false, 3>(m, q, chains, chain, rng_chain, iters, T0, alpha, key0, key1, swap_thr, srch, ws);
  }
}

template <int LG, int OBJ>
__global__ void __launch_bounds__(256) anneal_reg_h_kernel(DevModel m, QueuePtrs q, int chains, int iters, double T0,
                                                            double alpha, uint32_t key0, uint32_t key1,
                                                            uint64_t swap_thr, SearchParams srch, unsigned char *ws) {
  if (!gate_open(ws, m.gate, m.flags)) return;
  const int waves = blockDim.x >> 6;
  const int chain = uniform((int)blockIdx.x * waves + (int)(threadIdx.x >> 6));
  if (chain >= chains) return;
  anneal_reg_any<LG, OBJ>(m, q, chains, chain, (uint32_t)chain, iters, T0, alpha, key0, key1, swap_thr, srch, ws);
}

// ---- the joint order / batch-size search on small queues, state in registers ----
//
// Same register layout of the order; the layout is a 64-bit scalar mask of start flags
// (bit p set iff a batch begins at position p). The squeeze / delay / swap rules are the
// ones of plan_move taken on the mask (batch begin = highest flag at or below a position,
// batch end = next flag above it, or n; each lane's bounds are kept until a squeeze or delay
// changes the mask). The whole queue is one window of at most 64 positions: each lane
// gathers its batch's members with ds_bpermute, 8 or 16 offsets in flight at a time (pair
// terms), its TTFT is the prefill add-scan read at the batch's last lane plus the decode
// durations of the earlier batches, and the durations are a 32-bit max-scan confined to
// batches. Prefills, offsets and durations fit 32 bits (the fixed-size width checks); the
// timeline's prefix sums are plain 32-bit scans when the device check bounds it below 2^32, and
// saturate otherwise.

__host__ __device__ __forceinline__ bool reg_sized_fits(int n) { return n >= 1 && n <= 64; }

__device__ __forceinline__ int mask_begin(uint64_t fm, int p) {  // highest start at or below p
  const uint64_t le = p >= 63 ? fm : fm & ((uint64_t(2) << p) - 1);
  return 63 - __clzll(le);
}
__device__ __forceinline__ int mask_end(uint64_t fm, int n, int p) {  // first start above p, or n
  const uint64_t gt = p >= 63 ? 0ull : fm & ~((uint64_t(2) << p) - 1);
  return gt ? min(n, __builtin_ctzll(gt)) : n;
}

struct RegMove {
  bool made;
  int op, i, j, to, set0, clr0;
};

// plan_move on the mask (all wave-uniform)
__device__ __forceinline__ RegMove reg_plan(uint64_t fm, int n, int B, int op, int i, int j) {
  RegMove mv{false, op, i, j, i, -1, -1};
  if (op == 2) {
    mv.made = n >= 2;
    return mv;
  }
  const int s = mask_begin(fm, i), e = mask_end(fm, n, i);
  if (op == 0) {
    if (s == 0) return mv;
    const int sp = mask_begin(fm, s - 1);
    if (s - sp >= B) return mv;
    mv.made = true;
    mv.to = s;
    mv.clr0 = s;
    mv.set0 = s + 1 < e ? s + 1 : -1;
    return mv;
  }
  if (e == n) {
    if (e - s < 2) return mv;
    mv.made = true;
    mv.to = e - 1;
    mv.set0 = e - 1;
    return mv;
  }
  const int en = mask_end(fm, n, e);
  if (en - e >= B) return mv;
  mv.made = true;
  mv.to = e - 1;
  mv.set0 = e - 1;
  mv.clr0 = e;
  return mv;
}

__device__ __forceinline__ uint32_t bperm(uint32_t v, int src) {
  return (uint32_t)__builtin_amdgcn_ds_bpermute(src << 2, (int)v);
}

// Pair terms of W consecutive members of the lane's batch from offset d: all 2W ds_bpermute
// are in flight before their results are used.
template <int W>
__device__ __forceinline__ uint32_t pair_round(uint32_t L, uint32_t e, uint32_t d2, int b0, int bl, int d,
                                               uint32_t acc) {
  uint32_t Lj[W], ej[W];
#pragma unroll
  for (int u = 0; u < W; ++u) {
    const int src = min(b0 + d + u, kWave - 1);
    Lj[u] = bperm(L, src);
    ej[u] = bperm(e, src);
  }
#pragma unroll
  for (int u = 0; u < W; ++u) {
    const uint32_t mu = min(Lj[u], L);
    const uint32_t w = mad24_v(mu, mad24_v(d2, mu, ej[u]), 0u);
    acc += d + u < bl ? w : 0u;
  }
  return acc;
}

// Full replay of the order in registers with the batches given per lane by their first and
// last positions b0 <= lane <= b1 (lanes at or above n: b0 = b1 = lane), every batch at most
// maxb long: (met count, total latency). A member's TTFT is the sum of the prefills of every
// position up to its batch's end plus the decode durations of the earlier batches; its e2e
// adds its own decode time G after the batch prefill. Prefills, G and batch durations fit
// 32 bits (the host's width checks); the timeline need not: its prefix sums saturate at
// 2^32 - 1, which no threshold reaches, and the total latency is formed exactly as the sum of
// G, of each prefill times the requests from its batch's start onward and of each batch's
// decode duration times the requests after it.
// SAT = false: the whole timeline fits 32 bits (the host's check) and plain 32-bit scans do.
template <bool SAT>
__device__ __forceinline__ Score reg_replay_sized(const RegState &s, int b0, int b1, int maxb, int n, uint32_t d0,
                                                  uint32_t d2, int lane) {
  const bool valid = lane < n;
  const uint32_t L = s.A & 0xFFFFu, e = s.E & 0x3FFFFFFFu, kind = s.E >> 30;
  const int bl = b1 - b0 + 1;
  // prefills up to the batch's end: one add-scan read at the batch's last lane (the gather
  // is unconditional: ds_bpermute reads only lanes that execute it)
  const uint32_t pend = bperm(SAT ? scan_add_sat32(s.PF) : scan_add32(s.PF), b1);
  // pair terms: one round of gathers for batches of up to 8 (16 per round above)
  uint32_t acc = 0;
  if (maxb <= 8) {
    acc = pair_round<8>(L, e, d2, b0, bl, 0, 0u);
  } else {
    for (int d = 0; d < maxb; d += 16) acc = pair_round<16>(L, e, d2, b0, bl, d, acc);
  }
  const uint32_t G = valid ? __umul24(L, d0) + (acc >> 1) : 0u;
  // the batch's decode duration at its last lane
  const uint32_t D = seg_max32(G, b0, b1, lane);
  const bool last = valid && lane == b1;
  const uint32_t contrib = last ? D : 0u;
  uint32_t ttft, e2e, lo, hi;
  if constexpr (SAT) {
    // decode durations of the earlier batches: the inclusive scan moved up one lane
    const uint32_t SD =
        scan_add_sat32((uint32_t)__builtin_amdgcn_update_dpp(0, (int)contrib, kDppWaveShr1, 0xF, 0xF, false));
    ttft = add_sat(pend, SD);
    e2e = add_sat(ttft, G);
    // the latency sum in 16-bit halves (each lane below 2^23, each sum below 2^29)
    const uint32_t from = valid ? (uint32_t)(n - b0) : 0u, after = last ? (uint32_t)(n - 1 - b1) : 0u;
    lo = (G & 0xFFFFu) + (s.PF & 0xFFFFu) * from + (contrib & 0xFFFFu) * after;
    hi = (G >> 16) + (s.PF >> 16) * from + (contrib >> 16) * after;
  } else {
    ttft = pend + scan_add32(contrib) - contrib;
    e2e = ttft + G;
    // the latency sum: 16-bit halves of the 32-bit latencies, each sum below 2^22
    lo = valid ? (e2e & 0xFFFFu) : 0u;
    hi = valid ? (e2e >> 16) : 0u;
  }
  const bool met = valid && (kind == 0 ? ttft <= s.T : (kind == 2 ? e2e <= s.T : G <= s.T));
  const int64_t nmet = __popcll(__ballot(met));
  wave_all2<OpAdd, OpAdd>(lo, hi);
  return Score{nmet, (uint64_t)lo + ((uint64_t)hi << 16)};
}

template <int OBJ, bool SAT>
__device__ void anneal_reg_sized_body(const DevModel &m, const QueuePtrs &q, int chains, int chain,
                                      uint32_t rng_chain, int iters, double T0, double alpha, uint32_t key0,
                                      uint32_t key1, const SearchParams &srch, unsigned char *ws) {
  const int n = m.n, B = m.B;
  const int lane = lane_id();
  const uint32_t d0 = (uint32_t)m.d0, d2 = (uint32_t)m.d2;
  const WsHeader *h = reinterpret_cast<const WsHeader *>(ws);
  const int64_t t_ref = h->t_ref;
  const int64_t allmet = h->allmet;
  const uint16_t *start = reinterpret_cast<const uint16_t *>(ws + ws_off_start());
  const size_t stride = ws_perm_stride(n), fstride = ws_flag_stride(n);
  uint16_t *gbest = reinterpret_cast<uint16_t *>(ws + ws_off_best(n, chains)) + (size_t)chain * stride;
  uint16_t *gcur = reinterpret_cast<uint16_t *>(ws + ws_off_cur(n, chains)) + (size_t)chain * stride;
  uint8_t *gbest_f = ws + ws_off_best_starts(n, chains) + (size_t)chain * fstride;
  uint8_t *gcur_f = ws + ws_off_cur_starts(n, chains) + (size_t)chain * fstride;
  RegState cur{0u, 0u, 0u, 0u};
  const bool first = lane < n && lane % B == 0;
  uint64_t fm = __ballot(first);  // the maximum-size layout
  if (lane < n) {
    const uint32_t r = start[lane];
    const uint32_t lin = q.in_len[r], L = q.out_len[r], kind = q.kind[r], thr = q.thr[r];
    const uint32_t e = (uint32_t)(2 * (m.d1 + m.d2 * lin) + m.d2);
    const uint64_t thr_l = (uint64_t)thr * L;
    cur.A = L | (r << 16);
    cur.E = e | (kind << 30);
    cur.PF = (uint32_t)(m.p0 + m.p1 * lin);
    cur.T = kind == 1 ? (uint32_t)min(thr_l, (uint64_t)0xFFFFFFFFu) : thr;
    gbest[lane] = (uint16_t)r;
    gbest_f[lane] = first ? 1 : 0;
  }
  // each lane's batch bounds under the current layout (kept: swaps leave them unchanged)
  const int maxb = min(B, n);
  auto bounds = [&](uint64_t f, int &b0, int &b1) {
    b0 = lane < n ? mask_begin(f, lane) : lane;
    b1 = lane < n ? mask_end(f, n, lane) - 1 : lane;
  };
  int cb0, cb1;
  bounds(fm, cb0, cb1);
  const Score s0 = reg_replay_sized<SAT>(cur, cb0, cb1, maxb, n, d0, d2, lane);
  int64_t cn = s0.n;
  uint64_t ct = s0.t;
  int64_t bn = cn;
  uint64_t bt = ct;
  int64_t biter = -1, accepts = 0;
  uint64_t digest = kFnvOffset;
  Cooling cool{T0, alpha, srch.level_len, srch.level_len};
  SizedDraws ds;
  const int iters_run = (srch.early_exit && allmet) ? 0 : iters;
  for (int k = 0; k < iters_run; ++k) {
    if ((k & (kWave - 1)) == 0) ds.refill(k, lane, n, rng_chain, key0, key1);
    const uint32_t pk = ds.packed(k), w3 = ds.word3(k);
    const RegMove mv = reg_plan(fm, n, B, (int)(pk >> 20), (int)(pk & 1023u), (int)((pk >> 10) & 1023u));
    if (mv.made) {
      uint64_t fc = fm;
      int nb0 = cb0, nb1 = cb1;
      // a swap of i and j, or an insert from i to `to` (lanes [i, to) take x[lane + 1], or
      // lanes (to, i] take x[lane - 1])
      const int addr = move_src_addr(mv.op == 2, mv.i, mv.op == 2 ? mv.j : mv.to, lane);
      const RegState cand{from_lane(addr, cur.A), from_lane(addr, cur.E), from_lane(addr, cur.PF),
                          from_lane(addr, cur.T)};
      if (mv.op != 2) {
        if (mv.clr0 >= 0) fc &= ~(uint64_t(1) << mv.clr0);
        if (mv.set0 >= 0) fc |= uint64_t(1) << mv.set0;
        bounds(fc, nb0, nb1);
      }
      // a swap inside one batch changes no batch's members: the score is unchanged
      const bool same = mv.op == 2 && mask_begin(fm, mv.i) == mask_begin(fm, mv.j);
      const Score sc = same ? Score{cn, ct} : reg_replay_sized<SAT>(cand, nb0, nb1, maxb, n, d0, d2, lane);
      if (obj_accept<OBJ>(cn, ct, sc.n - cn, (int64_t)(sc.t - ct), t_ref, cool.T, w3)) {
        cur = cand;
        fm = fc;
        cb0 = nb0;
        cb1 = nb1;
        cn = sc.n;
        ct = sc.t;
        ++accepts;
        digest = (digest ^ (uint64_t)k) * kFnvPrime;
        digest = (digest ^ (uint64_t)cn) * kFnvPrime;
        digest = (digest ^ ct) * kFnvPrime;
        if (obj_better<OBJ>(cn, ct, bn, bt)) {
          bn = cn;
          bt = ct;
          biter = k;
          if (lane < n) {
            gbest[lane] = (uint16_t)(cur.A >> 16);
            gbest_f[lane] = (uint8_t)((fm >> lane) & 1u);
          }
        }
      }
    }
    cool.step();
  }
  if (lane < n) {
    gcur[lane] = (uint16_t)(cur.A >> 16);
    gcur_f[lane] = (uint8_t)((fm >> lane) & 1u);
  }
  if (lane == 0) write_record(ws, n, chain, cn, ct, bn, bt, biter, accepts, digest, allmet);
}

template <int OBJ>
__global__ void __launch_bounds__(256) anneal_reg_sized_kernel(DevModel m, QueuePtrs q, int chains, int iters,
                                                                double T0, double alpha, uint32_t key0, uint32_t key1,
                                                                SearchParams srch, unsigned char *ws) {
  if (!gate_open(ws, m.gate, m.flags)) return;
  const int waves = blockDim.x >> 6;
  const int chain = uniform((int)blockIdx.x * waves + (int)(threadIdx.x >> 6));
  if (chain >= chains) return;
  if (m.flags & kFlagTime32)
    anneal_reg_sized_body<OBJ, false>(m, q, chains, chain, (uint32_t)chain, iters, T0, alpha, key0, key1, srch, ws);
  else
    anneal_reg_sized_body<OBJ, true>(m, q, chains, chain, (uint32_t)chain, iters, T0, alpha, key0, key1, srch, ws);
}

// ---- the fitted latency model on small queues, state in registers ----
//
// A member's prefill and decode times depend only on its own lengths and its batch's size,
// so the replay needs no gathers: each lane takes its batch size from the flag mask and
// its two closed forms, in 32 bits when every member's time fits (else 64-bit closed forms,
// a 64-bit max-scan of (first position of the batch << 58 | time) and a 64-bit add-scan,
// every time below 2^57: the host's checks). Fixed-size batches take swap / insert
// proposals with the layout fixed; the batch-size search takes squeeze / delay / swap as
// above.

struct RegFit {
  uint32_t A;   // output length | request id << 16
  uint32_t LK;  // input length | kind << 16
  uint32_t T, T2;
};

// M32: every member's time fits 32 bits (the host's check). The closed forms then run in
// 32-bit arithmetic (exact: products wrap only inside ring expressions whose value fits), the
// batch starts in a saturating 32-bit scan (a start that saturates can meet no threshold,
// every threshold being below 2^32 - 1; T and T2 hold the thresholds of the decode-time
// tests already multiplied by l_out, saturated), and the total latency exactly as the sum of
// the member times plus each batch's duration times the number of requests after it.
template <bool M32>
__device__ __forceinline__ Score reg_replay_fit(const DevFit &f, const RegFit &s, uint64_t fm, int lane) {
  const int n = f.n;
  const bool valid = lane < n;
  const uint32_t kind = s.LK >> 16;
  const int b0 = valid ? mask_begin(fm, lane) : lane;
  const int b1 = valid ? mask_end(fm, n, lane) - 1 : lane;
  if constexpr (M32) {
    const uint32_t L = s.A & 0xFFFFu, l = s.LK & 0xFFFFu, b = (uint32_t)(b1 - b0 + 1);
    const uint32_t tp = (uint32_t)f.ap * b * l + (uint32_t)f.bp * b + (uint32_t)f.cp * l + (uint32_t)f.dp;
    const uint32_t td = L * ((uint32_t)f.bd * b + (uint32_t)f.dd) +
                        ((uint32_t)f.ad * b + (uint32_t)f.cd) * (L * l + ((L * (L + 1u)) >> 1));
    const uint32_t E = valid ? tp + td : 0u;
    const uint32_t D = seg_max32(E, b0, b1, lane);
    const bool last = valid && lane == b1;
    const uint32_t contrib = last ? D : 0u;
    // exclusive start: the inclusive scan of the contributions moved up one lane
    const uint32_t S = scan_add_sat32((uint32_t)__builtin_amdgcn_update_dpp(0, (int)contrib, kDppWaveShr1, 0xF, 0xF,
                                                                            false));
    const uint32_t ttft = add_sat(S, tp), e2e = add_sat(S, E);
    const bool met = valid && (kind == 0   ? ttft <= s.T
                               : kind == 1 ? td <= s.T
                               : kind == 2 ? e2e <= s.T
                                           : (ttft <= s.T && td <= s.T2));
    const int64_t nmet = __popcll(__ballot(met));
    // sum of e2e = sum of E + sum over batches of D * (requests after the batch), in 16-bit
    // halves (each lane below 2^22, each sum below 2^28)
    const uint32_t after = last ? (uint32_t)(n - 1 - b1) : 0u;
    uint32_t lo = (E & 0xFFFFu) + (contrib & 0xFFFFu) * after, hi = (E >> 16) + (contrib >> 16) * after;
    wave_all2<OpAdd, OpAdd>(lo, hi);
    return Score{nmet, (uint64_t)lo + ((uint64_t)hi << 16)};
  } else {
    const uint64_t L = s.A & 0xFFFFu, l = s.LK & 0xFFFFu;
    const uint64_t b = (uint64_t)(b1 - b0 + 1);
    const uint64_t tp = fit_prefill(f, b, l), td = fit_decode(f, b, l, L), E = tp + td;
    constexpr uint64_t kTimeMask = (uint64_t(1) << 58) - 1;
    const uint64_t D = scan_max64(valid ? ((uint64_t)b0 << 58) | E : 0ull) & kTimeMask;
    const uint64_t contrib = (valid && lane == b1) ? D : 0ull;
    const uint64_t S = scan_add64(contrib) - contrib;
    const uint64_t ttft = S + tp, e2e = S + E;
    const bool met = valid && fit_met(kind, s.T, s.T2, L, ttft, td, e2e);
    const int64_t nmet = __popcll(__ballot(met));
    return Score{nmet, wave_sum64_dpp(valid ? e2e : 0ull)};
  }
}

template <int OBJ, bool M32>
__device__ void anneal_reg_fit_body(const DevFit &f, const QueuePtrs &q, const uint32_t *thr2, int chains, int chain,
                                    uint32_t rng_chain, int iters, double T0, double alpha, uint32_t key0,
                                    uint32_t key1, uint64_t swap_thr, const SearchParams &srch, unsigned char *ws) {
  const int n = f.n, B = f.B;
  const bool search = f.policy == 2;
  const int lane = lane_id();
  const WsHeader *h = reinterpret_cast<const WsHeader *>(ws);
  const int64_t t_ref = h->t_ref;
  const int64_t allmet = h->allmet;
  const uint16_t *start = reinterpret_cast<const uint16_t *>(ws + ws_off_start());
  const size_t stride = ws_perm_stride(n), fstride = ws_flag_stride(n);
  uint16_t *gbest = reinterpret_cast<uint16_t *>(ws + ws_off_best(n, chains)) + (size_t)chain * stride;
  uint16_t *gcur = reinterpret_cast<uint16_t *>(ws + ws_off_cur(n, chains)) + (size_t)chain * stride;
  uint8_t *gbest_f = ws + ws_off_best_starts(n, chains) + (size_t)chain * fstride;
  uint8_t *gcur_f = ws + ws_off_cur_starts(n, chains) + (size_t)chain * fstride;
  RegFit cur{0u, 0u, 0u, 0u};
  const bool first = lane < n && lane % B == 0;
  uint64_t fm = __ballot(first);  // the maximum-size layout
  if (lane < n) {
    const uint32_t r = start[lane];
    cur.A = (uint32_t)q.out_len[r] | (r << 16);
    cur.LK = (uint32_t)q.in_len[r] | ((uint32_t)q.kind[r] << 16);
    cur.T = q.thr[r];
    cur.T2 = thr2 ? thr2[r] : 0u;
    if (M32) {
      // thresholds of the decode-time tests, multiplied by l_out and saturated
      const uint64_t L = q.out_len[r];
      if (q.kind[r] == 1) cur.T = (uint32_t)min((uint64_t)cur.T * L, (uint64_t)0xFFFFFFFFu);
      cur.T2 = (uint32_t)min((uint64_t)cur.T2 * L, (uint64_t)0xFFFFFFFFu);
    }
    gbest[lane] = (uint16_t)r;
    gbest_f[lane] = first ? 1 : 0;
  }
  const Score s0 = reg_replay_fit<M32>(f, cur, fm, lane);
  int64_t cn = s0.n;
  uint64_t ct = s0.t;
  int64_t bn = cn;
  uint64_t bt = ct;
  int64_t biter = -1, accepts = 0;
  uint64_t digest = kFnvOffset;
  Cooling cool{T0, alpha, srch.level_len, srch.level_len};
  SizedDraws ds;
  ProposalStream ps;
  const int iters_run = (srch.early_exit && allmet) ? 0 : iters;
  for (int k = 0; k < iters_run; ++k) {
    uint32_t w3;
    RegMove mv;
    if (search) {
      if ((k & (kWave - 1)) == 0) ds.refill(k, lane, n, rng_chain, key0, key1);
      const uint32_t pk = ds.packed(k);
      w3 = ds.word3(k);
      mv = reg_plan(fm, n, B, (int)(pk >> 20), (int)(pk & 1023u), (int)((pk >> 10) & 1023u));
    } else {
      if ((k & (kWave - 1)) == 0) ps.refill(k, lane, n, rng_chain, key0, key1, swap_thr, 0);
      const uint32_t pk = ps.packed(k);
      w3 = ps.word3(k);
      const int i = (int)(pk & 1023u), j = (int)((pk >> 10) & 1023u);
      // a fixed-size move: swap (op 2) or insert from i to j (op 3), layout unchanged
      mv = RegMove{true, ((pk >> 20) & 1u) ? 3 : 2, i, j, j, -1, -1};
    }
    if (mv.made) {
      uint64_t fc = fm;
      const int addr = move_src_addr(mv.op == 2, mv.i, mv.op == 2 ? mv.j : mv.to, lane);
      const RegFit cand{from_lane(addr, cur.A), from_lane(addr, cur.LK), from_lane(addr, cur.T), from_lane(addr, cur.T2)};
      if (mv.op != 2) {
        if (mv.clr0 >= 0) fc &= ~(uint64_t(1) << mv.clr0);
        if (mv.set0 >= 0) fc |= uint64_t(1) << mv.set0;
      }
      // a swap, or a fixed-layout insert, inside one batch keeps every member's batch size and
      // every batch's duration: the score is unchanged
      const bool same = mv.op >= 2 && mask_begin(fm, mv.i) == mask_begin(fm, mv.j);
      const Score sc = same ? Score{cn, ct} : reg_replay_fit<M32>(f, cand, fc, lane);
      if (obj_accept<OBJ>(cn, ct, sc.n - cn, (int64_t)(sc.t - ct), t_ref, cool.T, w3)) {
        cur = cand;
        fm = fc;
        cn = sc.n;
        ct = sc.t;
        ++accepts;
        digest = (digest ^ (uint64_t)k) * kFnvPrime;
        digest = (digest ^ (uint64_t)cn) * kFnvPrime;
        digest = (digest ^ ct) * kFnvPrime;
        if (obj_better<OBJ>(cn, ct, bn, bt)) {
          bn = cn;
          bt = ct;
          biter = k;
          if (lane < n) {
            gbest[lane] = (uint16_t)(cur.A >> 16);
            gbest_f[lane] = (uint8_t)((fm >> lane) & 1u);
          }
        }
      }
    }
    cool.step();
  }
  if (lane < n) {
    gcur[lane] = (uint16_t)(cur.A >> 16);
    gcur_f[lane] = (uint8_t)((fm >> lane) & 1u);
  }
  if (lane == 0) write_record(ws, n, chain, cn, ct, bn, bt, biter, accepts, digest, allmet);
}

template <int OBJ>
__global__ void __launch_bounds__(256) anneal_reg_fit_kernel(DevFit f, QueuePtrs q, const uint32_t *thr2, int chains,
                                                              int iters, double T0, double alpha, uint32_t key0,
                                                              uint32_t key1, uint64_t swap_thr, SearchParams srch,
                                                              unsigned char *ws) {
  if (!fit_gate_open(ws, f)) return;
  const int waves = blockDim.x >> 6;
  const int chain = uniform((int)blockIdx.x * waves + (int)(threadIdx.x >> 6));
  if (chain >= chains) return;
  if (f.m32)
    anneal_reg_fit_body<OBJ, true>(f, q, thr2, chains, chain, (uint32_t)chain, iters, T0, alpha, key0, key1, swap_thr,
                                   srch, ws);
  else
    anneal_reg_fit_body<OBJ, false>(f, q, thr2, chains, chain, (uint32_t)chain, iters, T0, alpha, key0, key1, swap_thr,
                                    srch, ws);
}

}  // namespace sa
