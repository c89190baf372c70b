// Annealing chains under static admission, one batch per wave (33 <= B <= 64), with the SLO
// limit of every member held in registers; for queues whose whole timeline fits 32 bits.
//
// The delta re-simulation is that of the one-batch-per-wave kernel: a move changes the
// members of batches a..c by one leaving request o and one joining request e each, and the
// later batches only shift. The met counts are kept another way. Row k of a register array
// holds, lane by lane, the limits of batch k's members: a member meets its SLO iff its
// batch starts before its limit (thr + 1 - P for TTFT with P the batch prefill, thr + 1 - F
// for end-to-end with F its finish offset, all or nothing for TPOT, whose time per output
// token does not depend on the start; the staged records hold thr + 1 and the kind as flag
// bits above e). A changed batch rewrites its row; each proposal then counts the met
// members of every row at its candidate start with one compare and one population count
// per row. No batch needs bounds on the starts that keep its flags, and no shifted batch
// is recounted member by member. A row is a set: only its count is read, and a changed
// batch rewrites all of it, so which lane holds which member does not matter.
//
// Per changed batch one three-way reduction gives the newcomer's pair-cost sum, the change
// of the staying members' finish offsets (for the latency delta) and their largest new
// offset; the new duration is the larger of that and the newcomer's offset. A rejected
// proposal restores the offsets as the other kernel does and rebuilds the rows of the
// changed batches from the restored offsets and the old prefills.
//
// Widths: those of the one-batch-per-wave kernel, and every time on the timeline of any
// order below 2^32 - 2 (a device check), so starts and limits are u32 and a TPOT member that
// meets its SLO has the limit 2^32 - 1, above every start.
#pragma once
#include "anneal_wave.h"
#include "anneal_sized.h"

namespace sa {

// The limit rows: one vector value of MR registers. A row picked by a wave-uniform index is
// written with one indexed register move; rows picked by constants are plain registers.
template <int MR>
using LimRows = uint32_t __attribute__((ext_vector_type(MR)));

// Number of limit rows for M batches (the kernel is instantiated for these).
__host__ __device__ constexpr int limit_rows_for(int M) { return M <= 8 ? 8 : (M <= 16 ? 16 : 32); }

// Members meeting their SLO: row u at the start in lane u of S.
template <int MR>
__device__ __forceinline__ int64_t rows_met(const LimRows<MR> &lim, uint32_t S) {
  uint32_t cnt = 0;
  static_for<MR>([=, &lim, &cnt](auto uc) __attribute__((always_inline)) {
    constexpr int u = decltype(uc)::value;
    cnt += (uint32_t)__popcll(__ballot(readlane(S, u) < lim[u]));
  });
  return (int64_t)cnt;
}

// The limit of a member from its record's third word z (e | 2^30 for end-to-end | 2^31 for
// TPOT, TTFT with neither) and thr1 = threshold + 1: met iff the batch starts before it.
// TTFT: thr1 - P, end-to-end: thr1 - F (0 when not positive: never met), TPOT: 2^32 - 1 when
// F - P < thr1, else 0. The zero spare record gives 0.
__device__ __forceinline__ uint32_t limit_of(uint32_t z, uint32_t thr1, uint32_t P, uint32_t F) {
  const uint32_t off = z < (1u << 30) ? P : F;
  const uint32_t by_start = __builtin_elementwise_sub_sat(thr1, off);
  const uint32_t tpot = F - P < thr1 ? 0xFFFFFFFFu : 0u;
  return (int32_t)z < 0 ? tpot : by_start;
}

// batch records, lane k = batch k: start, prefill, duration
struct RowRecs {
  uint32_t S, P, D;
};

// LDS of one chain: the order padded with 64 spare ids n (read by lanes past the last
// batch), finish offsets (n + 2 entries), 48 bytes of proposal table per batch.
__host__ __device__ __forceinline__ size_t rows_chain_bytes(int n, int B) {
  const size_t M = (size_t)(n + B - 1) / B;
  return (((size_t)(n + 64) * 2 + 15) & ~size_t(15)) + (((size_t)(n + 2) * 4 + 15) & ~size_t(15)) + M * 48;
}

struct RowChain {
  const uint4 *req;
  uint16_t *perm;  // the order, n entries and 64 spare ids n
  uint32_t *F;     // n + 2 entries: F[n] is read and written by lanes past a batch
  uint4 *tab;      // 3 entries per batch, written by the prologue for changed batches
  uint32_t d0, d2;
  uint32_t vd2;  // d2 in a vector register (an operand of the vector multiply-adds)
  int N, B, M, lane;
  RowRecs cur, cand;
  uint32_t fo, ovec;  // lane k: old F and id of the leaving member of changed batch k

  __device__ __forceinline__ int batch_size(int k) const { return min(B, N - k * B); }
  __device__ __forceinline__ int64_t requests_in(int k0, int k1) const {
    return k1 <= k0 ? 0 : (int64_t)min(N, k1 * B) - (int64_t)k0 * B;
  }
};

// Full evaluation of the current order: F, the limit rows and the batch records; returns
// (n, t).
template <int MR>
__device__ __forceinline__ Score rows_init(RowChain &c, LimRows<MR> &lim) {
  const int lane = c.lane;
  if (lane == 0) {
    c.F[c.N] = 0u;
    c.F[c.N + 1] = 0u;
  }
  lim = LimRows<MR>(0u);
  wave_sync_lds();
  uint32_t carry = 0;
  uint64_t tl = 0;
  c.cur = RowRecs{0, 0, 0};
  for (int k = 0; k < c.M; ++k) {
    const int q0 = k * c.B;
    const int bs = c.batch_size(k);
    const bool valid = lane < bs;
    const int r = valid ? (int)c.perm[q0 + lane] : c.N;
    const uint4 rq = c.req[r];
    const uint32_t L = rq.x >> 16;
    uint32_t P = 0, acc = 0;
    for (int jj = 0; jj < bs; ++jj) {
      const uint4 o = c.req[c.perm[q0 + jj]];
      P += o.w;
      acc += w2(o.x >> 16, rec_e<true>(o.z), L, c.d2);
    }
    const uint32_t Fv = valid ? P + __umul24(L, c.d0) + (acc >> 1) : 0u;
    if (valid) c.F[r] = Fv;
    const uint64_t SF = Seg<6>::sum_wide(Fv, lane);
    const uint32_t D = Seg<6>::template all<OpMax>(Fv, lane);
    lim[k] = valid ? limit_of(rq.z, rq.y, P, Fv) : 0u;
    c.cur.S = lane == k ? carry : c.cur.S;
    c.cur.P = lane == k ? P : c.cur.P;
    c.cur.D = lane == k ? D : c.cur.D;
    tl += (uint64_t)bs * carry + SF;
    carry += D;
  }
  wave_sync_lds();
  return Score{rows_met(lim, c.cur.S), tl};
}

// Candidate of changed batch k starting `shift` later: the new finish offsets (written to F),
// its limit row and record, and the latency change. Returns the duration change.
template <int MR>
__device__ __forceinline__ int64_t rows_changed(RowChain &c, LimRows<MR> &lim, int k, int64_t shift, int64_t &dt) {
  const int lane = c.lane, N = c.N;
  const int bs = c.batch_size(k);
  const bool valid = lane < bs;
  const uint4 t0 = c.tab[3 * k], t1 = c.tab[3 * k + 1], t2 = c.tab[3 * k + 2];
  const uint32_t o = t0.x, e = t0.y, Lo = t0.z, eo = t0.w;
  uint32_t Le = t1.x, ee = t1.y;
  const uint32_t dP = t1.z;
  const uint32_t FeBase = t2.x;
  uint32_t kinde = t2.y, thre = t2.z, Pc = t2.w;
  // operands of vector instructions only: kept in the vector registers the broadcast read
  // filled (as wave-uniform values they would be moved to scalar registers and back)
  asm volatile("" : "+v"(Le), "+v"(ee), "+v"(kinde), "+v"(thre), "+v"(Pc));
  // lanes past the batch take the spare id n (their read of the order, which stays inside
  // it thanks to the 64 spare entries, is discarded), the zero spare record and F[n],
  // whatever it holds, and write F[n] back: nothing they compute reaches a result (their
  // sums and maxima are masked out and the spare record's limit is 0 whatever the offset)
  const uint32_t rr = c.perm[k * c.B + lane];
  const uint32_t r = valid ? rr : (uint32_t)N;
  const uint4 rq = c.req[r];
  const uint32_t Fm = c.F[r];
  const uint32_t Lm = rq.x >> 16, em = rec_e<true>(rq.z);
  const uint32_t mue = min(Lm, Le), muo = min(Lm, Lo);
  const uint32_t te = vmul24(mue, vmad24(c.vd2, mue, em));   // w(m, e)
  const uint32_t wem = vmul24(mue, vmad24(c.vd2, mue, ee));  // w(e, m)
  const uint32_t wom = vmul24(muo, vmad24(c.vd2, muo, eo));  // w(o, m)
  const int32_t dwh = (int32_t)(wem - wom) >> 1;
  const bool is_out = r == o;
  const bool stay = valid && !is_out;
  const uint32_t Fs = Fm + dP + (uint32_t)dwh;
  uint32_t tsum = te, dsum = stay ? (uint32_t)dwh : 0u, dmax = stay ? Fs : 0u;
  wave_all3<OpAdd, OpAdd, OpMax>(tsum, dsum, dmax);
  const uint32_t Fe = FeBase + (tsum >> 1);
  const uint32_t Dn = max(dmax, Fe);
  const uint32_t Fc = is_out ? Fe : Fs;
  c.F[is_out ? e : r] = Fc;
  // lanes past the batch hold the spare record: limit 0
  const uint32_t z = is_out ? kinde : rq.z, thr1 = is_out ? thre : rq.y;
  lim[k] = limit_of(z, thr1, Pc, Fc);
  const uint32_t S = readlane(c.cur.S, k) + (uint32_t)shift;
  const uint32_t D0 = readlane(c.cur.D, k), Fo = readlane(c.fo, k);
  c.cand.S = wlane_m0(S, k, c.cand.S);
  c.cand.D = wlane_m0(Dn, k, c.cand.D);
  const int64_t dSF =
      (int64_t)(bs - 1) * (int64_t)(int32_t)rfl(dP) + (int64_t)(int32_t)dsum + ((int64_t)Fe - (int64_t)Fo);
  dt += (int64_t)bs * shift + dSF;
  return (int64_t)Dn - (int64_t)D0;
}

// Batches [k0, k1) keep their members and start `shift` later.
__device__ __forceinline__ void rows_shift(RowChain &c, int k0, int k1, int64_t shift, int64_t &dt) {
  const bool in = c.lane >= k0 && c.lane < k1;
  c.cand.S = in ? c.cur.S + (uint32_t)shift : c.cand.S;
  dt += shift * c.requests_in(k0, k1);
}

// Scores a move that changes batches (a < c): fills cand and the rows of the changed
// batches, returns the candidate met count and adds the latency change to dt.
template <int MR>
__device__ __forceinline__ int64_t rows_propose(RowChain &c, LimRows<MR> &lim, const Move &mv, int64_t &dt) {
  c.cand = c.cur;
  wave_prologue<true>(c.req, c.perm, c.F, c.tab, c.d0, c.d2, c.M, c.B, c.lane, c.cur.P, mv, c.fo, c.ovec, c.cand.P);
  dt = 0;
  int64_t carry = rows_changed(c, lim, mv.a, 0, dt);
  const int64_t shift_mid = carry;  // start change of the batches between a and c (swap)
  if (mv.type == 2) {
    for (int k = mv.a + 1; k <= mv.c; ++k) carry += rows_changed(c, lim, k, carry, dt);
  } else {
    if (mv.c > mv.a + 1) rows_shift(c, mv.a + 1, mv.c, shift_mid, dt);
    carry += rows_changed(c, lim, mv.c, shift_mid, dt);
  }
  if (carry != 0 && mv.c + 1 < c.M) rows_shift(c, mv.c + 1, c.M, carry, dt);
  return rows_met(lim, c.cand.S);
}

// Restores F and the limit rows after a rejected proposal.
template <int MR>
__device__ __forceinline__ void rows_undo(RowChain &c, LimRows<MR> &lim, const Move &mv) {
  const int lane = c.lane, N = c.N;
  for (int k = mv.a; k <= mv.c; ++k) {
    if (mv.type == 1 && k != mv.a && k != mv.c) continue;
    const bool valid = lane < c.batch_size(k);
    const uint4 t0 = c.tab[3 * k], t1 = c.tab[3 * k + 1];
    const uint32_t o = t0.x, Lo = t0.z, eo = t0.w, Le = t1.x, ee = t1.y, dP = t1.z;
    // as in rows_changed, lanes past the batch work on F[n]; the leaving member's lane
    // restores its own slot (which the newcomer's offset of another batch may hold)
    const uint32_t rr = c.perm[k * c.B + lane];
    const uint32_t r = valid ? rr : (uint32_t)N;
    const uint4 rq = c.req[r];
    const uint32_t Fm = c.F[r];
    const uint32_t Lm = rq.x >> 16;
    const uint32_t mue = min(Lm, Le), muo = min(Lm, Lo);
    const uint32_t wem = vmul24(mue, vmad24(c.vd2, mue, ee));
    const uint32_t wom = vmul24(muo, vmad24(c.vd2, muo, eo));
    const int32_t dwh = (int32_t)(wem - wom) >> 1;
    const bool is_out = r == o;
    const uint32_t Fold = is_out ? readlane(c.fo, k) : Fm - dP - (uint32_t)dwh;
    c.F[r] = Fold;
    lim[k] = limit_of(rq.z, rq.y, readlane(c.cur.P, k), Fold);
  }
  wave_sync_lds();
}

// One chain by one wave: record slot `chain`, Philox chain index `rng_chain`, the request
// records in `req`, the chain's LDS at `wb`.
// OBJ: objective (0 attainment, then total latency; 1 ratio n / t).
template <int OBJ, int MR>
__device__ void anneal_rows_body(const DevModel &m, const StaticParams &sp, const uint4 *req, unsigned char *wb,
                                 int chains, int chain, uint32_t rng_chain, int iters, double T0, double alpha,
                                 uint32_t key0, uint32_t key1, uint64_t swap_thr, const SearchParams &srch,
                                 unsigned char *ws) {
  const int n = m.n, B = m.B;
  const size_t perm_b = ((size_t)(n + 64) * 2 + 15) & ~size_t(15);
  const size_t f_b = ((size_t)(n + 2) * 4 + 15) & ~size_t(15);
  const int lane = lane_id();
  RowChain st;
  st.req = req;
  st.perm = reinterpret_cast<uint16_t *>(wb);
  st.F = reinterpret_cast<uint32_t *>(wb + perm_b);
  st.tab = reinterpret_cast<uint4 *>(wb + perm_b + f_b);
  st.d0 = sp.d0;
  st.d2 = sp.d2;
  st.vd2 = sp.d2;
  asm volatile("" : "+v"(st.vd2));
  st.N = n;
  st.B = B;
  st.M = (n + B - 1) / B;
  st.lane = lane;
  st.fo = 0u;
  st.ovec = 0u;
  LimRows<MR> lim;
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
  st.perm[n + lane] = (uint16_t)n;
  wave_sync_lds();
  const Score s0 = rows_init(st, lim);
  int64_t cn = s0.n;
  uint64_t ct = s0.t;
  int64_t bn = cn;
  uint64_t bt = ct;
  int64_t biter = -1, accepts = 0;
  uint64_t digest = kFnvOffset;
  Cooling cool{T0, alpha, srch.level_len, srch.level_len};
  ProposalStream ps;  // at most 32 batches: the batch indices travel with the move
  const int iters_run = (srch.early_exit && allmet) ? 0 : iters;
  for (int k = 0; k < iters_run; ++k) {
    if ((k & (kWave - 1)) == 0) ps.refill(k, lane, n, rng_chain, key0, key1, swap_thr, sp.bmagic);
    const uint32_t pk = ps.packed(k), w3 = ps.word3(k);
    const int i = (int)(pk & 1023u), j = (int)((pk >> 10) & 1023u);
    Move mv;
    mv.type = (int)((pk >> 20) & 1u) + 1;
    mv.i = i;
    mv.j = j;
    mv.a = (int)((pk >> 21) & 31u);
    mv.c = (int)(pk >> 26);
    bool acc;
    if (mv.a == mv.c) {
      // same batch: every batch keeps its members, the objective is unchanged
      acc = true;
      apply_move_lds(st.perm, mv.type, i, j, lane);
    } else {
      int64_t dt;
      const int64_t nn = rows_propose(st, lim, mv, dt);
      acc = obj_accept<OBJ>(cn, ct, nn - cn, dt, t_ref, cool.T, w3);
      if (acc) {
        apply_move_lds(st.perm, mv.type, i, j, lane);
        st.cur = st.cand;
        cn = nn;
        ct += (uint64_t)dt;
      } else {
        rows_undo(st, lim, mv);
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

// One wave per chain; blockDim / 64 chains per workgroup; MR >= the number of batches.
template <int OBJ, int MR>
__global__ void __launch_bounds__(1024) anneal_rows_kernel(DevModel m, StaticParams sp, QueuePtrs q, int chains,
                                                           int iters, double T0, double alpha, uint32_t key0,
                                                           uint32_t key1, uint64_t swap_thr, SearchParams srch,
                                                           unsigned char *ws) {
  extern __shared__ __align__(16) unsigned char lds[];
  if (!gate_open(ws, m.gate, m.flags)) return;
  const int n = m.n;
  const int waves = blockDim.x >> 6;
  uint4 *req = reinterpret_cast<uint4 *>(lds);
  const int wave = uniform((int)(threadIdx.x >> 6));
  unsigned char *wb = lds + (size_t)(n + 1) * 16 + (size_t)wave * rows_chain_bytes(n, m.B);
  load_static_records(q, m, req);
  __syncthreads();
  // thresholds as thr1 = threshold + 1 (a TPOT product above 2^32 - 2 is first lowered to
  // 2^32 - 2, which decides alike: F - P stays below 2^32 - 1), and the kind as flag bits
  // above e (e | 2^30 for end-to-end | 2^31 for TPOT; e < 2^24 by the width checks); the
  // spare record keeps 0
  for (int r = threadIdx.x; r < n; r += blockDim.x) {
    const uint4 v = req[r];
    const uint32_t kind = v.z & 3u;
    req[r].y = min(v.y, 0xFFFFFFFEu) + 1u;
    req[r].z = (v.z >> 2) | (kind == 2u ? 1u << 30 : 0u) | (kind == 1u ? 1u << 31 : 0u);
  }
  __syncthreads();
  const int chain = uniform((int)blockIdx.x * waves + wave);
  if (chain >= chains) return;
  anneal_rows_body<OBJ, MR>(m, sp, req, wb, chains, chain, (uint32_t)chain, iters, T0, alpha, key0, key1, swap_thr,
                            srch, ws);
}

}  // namespace sa
