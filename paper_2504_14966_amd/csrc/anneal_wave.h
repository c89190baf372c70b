// Annealing chains under static admission when one batch fills one wave (33 <= B <= 64).
//
// Same delta re-simulation as the row kernel (a move changes the membership of batches
// a..c by one leaving request o and one joining request e each; later batches only shift),
// laid out for a batch per wave:
//   - the batch records (start, prefill, duration, met count, slack bounds) live in vector
//     registers, lane k holding batch k (at most 32 batches), so reading a record is a
//     v_readlane and shifting a range of batches is one lane-parallel update;
//   - at the start of a proposal one lane-parallel pass computes, for every changed batch,
//     o and e, their request fields, the prefill change, the newcomer's finish offset up to
//     its pair-cost sum, and the leaving member's old finish offset, and leaves them in a
//     48-byte LDS entry per batch; each changed batch then reads its entry as a broadcast;
//   - the newcomer's pair-cost sum is reduced over the current members and corrected by
//     w(e, e) - w(o, e), so no lane swaps its request before the reduction;
//   - the change of the sum of finish offsets, needed for the latency delta, is
//     (size - 1) * dP + sum over staying members of half their pair-cost change + Fe - Fo
//     (|sum| < 2^31 because B * max w < 2^32 is a host condition of this path).
// A rejected proposal restores staying members by the reverse update and every leaving
// member from the old value kept by the prologue.
#pragma once
#include "anneal_static.h"

namespace sa {

// 24-bit vector multiply(-add): operands below 2^24, results below 2^32
__device__ __forceinline__ uint32_t vmad24(uint32_t a, uint32_t b, uint32_t c) {
  uint32_t d;
  asm("v_mad_u32_u24 %0, %1, %2, %3" : "=v"(d) : "v"(a), "v"(b), "v"(c));
  return d;
}
__device__ __forceinline__ uint32_t vmul24(uint32_t a, uint32_t b) {
  uint32_t d;
  asm("v_mul_u32_u24 %0, %1, %2" : "=v"(d) : "v"(a), "v"(b));
  return d;
}
__device__ __forceinline__ uint32_t rfl(uint32_t v) { return (uint32_t)__builtin_amdgcn_readfirstlane((int)v); }

// Whole-wave all-reduces of two or three values at once, step by step, so that the DPP
// steps of one fill the wait states the other needs between dependent steps. The result
// is read from lane 63 into a scalar register.
template <class Op>
__device__ __forceinline__ uint32_t dpp_step(uint32_t v, int step) {
  switch (step) {
    case 0: return Op::f(v, dpp<kQuadXor1>(v));
    case 1: return Op::f(v, dpp<kQuadXor2>(v));
    case 2: return Op::f(v, dpp<kRowHalfMirror>(v));
    case 3: return Op::f(v, dpp<kRowMirror>(v));
    // rows 1 and 3 take the last lane of rows 0 and 2, then rows 2 and 3 the last lane of row 1
    case 4: return Op::f(v, (uint32_t)__builtin_amdgcn_update_dpp((int)Op::identity, (int)v, 0x142, 0xA, 0xF, false));
    default: return Op::f(v, (uint32_t)__builtin_amdgcn_update_dpp((int)Op::identity, (int)v, 0x143, 0xC, 0xF, false));
  }
}
template <class O1, class O2>
__device__ __forceinline__ void wave_all2(uint32_t &a, uint32_t &b) {
#pragma unroll
  for (int s = 0; s < 6; ++s) {
    a = dpp_step<O1>(a, s);
    b = dpp_step<O2>(b, s);
  }
  a = readlane(a, 63);
  b = readlane(b, 63);
}
template <class O1, class O2, class O3>
__device__ __forceinline__ void wave_all3(uint32_t &a, uint32_t &b, uint32_t &c) {
#pragma unroll
  for (int s = 0; s < 6; ++s) {
    a = dpp_step<O1>(a, s);
    b = dpp_step<O2>(b, s);
    c = dpp_step<O3>(c, s);
  }
  a = readlane(a, 63);
  b = readlane(b, 63);
  c = readlane(c, 63);
}

// Request records whose third word holds e above the kind (e << 2 | kind, KTOP false) or e
// below flag bits for the kind (e | 2^30 for end-to-end | 2^31 for TPOT, KTOP true): e, and
// the kind code a newcomer's entry carries (the kind, or the whole word).
template <bool KTOP>
__device__ __forceinline__ uint32_t rec_e(uint32_t z) {
  return KTOP ? (z & 0x3FFFFFFFu) : (z >> 2);
}
template <bool KTOP>
__device__ __forceinline__ uint32_t rec_kind_code(uint32_t z) {
  return KTOP ? z : (z & 3u);
}

// Lane-parallel setup of the changed batches of a move, lane k = batch k with prefill Pk:
// for each changed batch the leaving request o and the joining request e, their fields, the
// prefill change, w(e, e) - w(o, e) and the newcomer's finish offset up to half its pair-cost
// sum over the current members, written as three 16-byte entries of `tab`; fo and ovec take
// o's old finish offset and id, Pn the batch's prefill after the move.
template <bool KTOP = false>
__device__ __forceinline__ void wave_prologue(const uint4 *req, const uint16_t *perm, const uint32_t *F, uint4 *tab,
                                              uint32_t d0, uint32_t d2, int M, int B, int lane, uint32_t Pk,
                                              const Move &mv, uint32_t &fo, uint32_t &ovec, uint32_t &Pn) {
  const int k = lane;
  const bool chg = k < M && mv.changes(k);
  int opos, epos;
  if (mv.type == 1) {
    const int lo = min(mv.i, mv.j), hi = max(mv.i, mv.j);
    opos = k == mv.a ? lo : hi;
    epos = k == mv.a ? hi : lo;
  } else if (mv.i < mv.j) {  // insert moving right: each batch passes its first member left
    opos = k == mv.a ? mv.i : k * B;
    epos = k == mv.c ? mv.i : (k + 1) * B;
  } else {  // insert moving left: each batch passes its last member right
    opos = k == mv.c ? mv.i : (k + 1) * B - 1;
    epos = k == mv.a ? mv.i : k * B - 1;
  }
  if (!chg) {
    opos = 0;
    epos = 0;
  }
  const uint32_t o = perm[opos], e = perm[epos];
  const uint4 ro = req[o], re = req[e];
  fo = F[o];
  ovec = o;
  const uint32_t Lo = ro.x >> 16, eo = rec_e<KTOP>(ro.z), Le = re.x >> 16, ee = rec_e<KTOP>(re.z);
  const uint32_t dP = re.w - ro.w;
  const uint32_t Pc = Pk + dP;
  Pn = chg ? Pc : Pk;
  const uint32_t corr = w2(Le, ee, Le, d2) - w2(Lo, eo, Le, d2);  // w(e, e) - w(o, e)
  // the newcomer's offset up to half its pair-cost sum over the current members: every
  // pair cost mu (e_j + d2 mu) = 2 mu (d1 + d2 l_j) + d2 mu (mu + 1) is even, so that sum
  // and corr halve exactly one by one (corr as a signed value, |corr| < 2^31)
  const uint32_t FeBase = Pc + __umul24(Le, d0) + (uint32_t)((int32_t)corr >> 1);
  if (chg) {
    tab[3 * k] = make_uint4(o, e, Lo, eo);
    tab[3 * k + 1] = make_uint4(Le, ee, dP, corr);
    tab[3 * k + 2] = make_uint4(FeBase, rec_kind_code<KTOP>(re.z), re.y, Pc);
  }
  wave_sync_lds();
}

// batch records, lane k = batch k
struct LaneRecs {
  uint32_t Slo, Shi, P, D, cnt, A, Bv;
};

struct WaveChain {
  const uint4 *req;
  uint16_t *perm;  // the order, n entries
  uint32_t *F;     // n + 2 entries: F[n] = 0 is read by lanes past a batch, F[n + 1] takes their writes
  uint4 *tab;      // 3 entries per batch, written by the prologue for changed batches
  uint32_t d0, d2;
  int N, B, M, lane;
  LaneRecs cur, cand;
  uint32_t fo, ovec;  // lane k: old F and id of the leaving member of changed batch k

  __device__ __forceinline__ int batch_size(int k) const { return min(B, N - k * B); }
  __device__ __forceinline__ int64_t requests_in(int k0, int k1) const {
    return k1 <= k0 ? 0 : (int64_t)min(N, k1 * B) - (int64_t)k0 * B;
  }
  __device__ __forceinline__ uint64_t start_of(const LaneRecs &R, int k) const {
    return ((uint64_t)readlane(R.Shi, k) << 32) | readlane(R.Slo, k);
  }
  __device__ __forceinline__ void put(LaneRecs &R, int k, uint64_t S, uint32_t P, uint32_t D, uint32_t cnt,
                                      uint32_t A, uint32_t Bv) const {
    // written as other ? old : new so that a scalar new value is the select's first operand
    const bool other = lane != k;
    R.Slo = other ? R.Slo : (uint32_t)S;
    R.Shi = other ? R.Shi : (uint32_t)(S >> 32);
    R.P = other ? R.P : P;
    R.D = other ? R.D : D;
    R.cnt = other ? R.cnt : cnt;
    R.A = other ? R.A : A;
    R.Bv = other ? R.Bv : Bv;
  }

  // v_writelane of a wave-uniform value into lane k (lane select in m0, so that the value's
  // scalar register is the instruction's one scalar operand); k comes from the scalar unit.
  static __device__ __forceinline__ uint32_t wlane(uint32_t v, int k, uint32_t old) {
    asm volatile("v_writelane_b32 %0, %1, m0" : "=v"(old) : "s"(v), "{m0}"(k), "0"(old));
    return old;
  }

  // SLO flags of the members at start S (TTFT and end-to-end members are met iff
  // S <= thr - offset; TPOT members do not depend on S), the met count and the bounds
  // [Bv, A] of starts that keep every flag.
  // Per lane: the contribution to A (min) and Bv (max); returns the met count.
  __device__ __forceinline__ uint32_t slo(bool valid, uint32_t kind, uint32_t thr, uint32_t P, uint32_t Fv, uint64_t S,
                                          uint32_t &a_in, uint32_t &b_in) const {
    // thresholds are at most 2^32 - 2, so a start of 2^32 or more compares like 2^32 - 1
    // (plain logical operations, no short-circuit: the vector code needs no branches)
    const uint32_t S32 = (S >> 32) ? 0xFFFFFFFFu : (uint32_t)S;
    const bool tpot = kind == 1u;
    const bool tpot_ok = Fv - P <= thr;
    const uint32_t off = kind == 0u ? P : Fv;
    const uint32_t sl = thr - off;
    // flex: a TTFT or end-to-end member whose offset alone does not exceed the threshold,
    // met iff S <= sl; a TPOT member is met iff tpot_ok, whatever S
    const bool flex = valid & !tpot & !(off > thr);
    const bool in = S32 <= sl;
    const bool met = (flex & in) | (valid & tpot & tpot_ok);
    a_in = (flex & in) ? sl : 0xFFFFFFFFu;
    b_in = (flex & !in) ? sl + 1u : 0u;
    return (uint32_t)__popcll(__ballot(met));
  }

  // Full evaluation of the current order (pairwise closed form per batch).
  __device__ Score init() {
    if (lane == 0) {
      F[N] = 0u;
      F[N + 1] = 0u;
    }
    wave_sync_lds();
    uint64_t carry = 0, tl = 0;
    int64_t nmet = 0;
    cur = LaneRecs{0, 0, 0, 0, 0, 0, 0};
    for (int k = 0; k < M; ++k) {
      const int q0 = k * B;
      const int bs = batch_size(k);
      const bool valid = lane < bs;
      const int r = valid ? (int)perm[q0 + lane] : N;
      const Req rq = load_req(req, r);
      uint32_t P = 0, acc = 0;
      for (int jj = 0; jj < bs; ++jj) {
        const Req o = load_req(req, perm[q0 + jj]);
        P += o.pf;
        acc += w2(o.L, o.e, rq.L, d2);
      }
      const uint32_t Fv = valid ? P + __umul24(rq.L, d0) + (acc >> 1) : 0u;
      if (valid) F[r] = Fv;
      const uint64_t SF = Seg<6>::sum_wide(Fv, lane);
      uint32_t D = Fv, A, Bv;
      const uint32_t cnt = slo(valid, rq.kind, rq.thr, P, Fv, carry, A, Bv);
      wave_all3<OpMax, OpMin, OpMax>(D, A, Bv);
      put(cur, k, carry, P, D, cnt, A, Bv);
      tl += (uint64_t)bs * carry + SF;
      nmet += cnt;
      carry += D;
    }
    wave_sync_lds();
    return Score{nmet, tl};
  }

  // Lane-parallel setup of the changed batches of a move (lane k = batch k).
  __device__ void prologue(const Move &mv) {
    uint32_t Pn;
    wave_prologue(req, perm, F, tab, d0, d2, M, B, lane, cur.P, mv, fo, ovec, Pn);
  }

  // Candidate of changed batch k starting `shift` later: finish offsets (written to F),
  // record, met-count and latency changes. Returns the duration change.
  __device__ int64_t changed_row(int k, int64_t shift, int64_t &dn, int64_t &dt) {
    const int bs = batch_size(k);
    const bool valid = lane < bs;
    const uint4 t0 = tab[3 * k], t1 = tab[3 * k + 1], t2 = tab[3 * k + 2];
    const uint32_t o = t0.x, e = t0.y, Lo = t0.z, eo = t0.w;
    const uint32_t Le = t1.x, ee = t1.y, dP = t1.z;
    const uint32_t FeBase = t2.x, kinde = t2.y, thre = t2.z, Pc = t2.w;
    // lanes past the batch read the zero spare record and F[n] = 0 (their position is
    // clamped into the order and the read discarded, so that the row has no branch)
    const uint32_t r = valid ? (uint32_t)perm[min(k * B + lane, N - 1)] : (uint32_t)N;
    const uint4 rq = req[r];
    const uint32_t Fm = F[r];
    const uint32_t Lm = rq.x >> 16, em = rq.z >> 2;
    const uint32_t mue = min(Lm, Le), muo = min(Lm, Lo);
    const uint32_t te = vmul24(mue, vmad24(d2, mue, em));   // w(m, e)
    const uint32_t wem = vmul24(mue, vmad24(d2, mue, ee));  // w(e, m)
    const uint32_t wom = vmul24(muo, vmad24(d2, muo, eo));  // w(o, m)
    const int32_t dwh = (int32_t)(wem - wom) >> 1;
    const bool is_out = r == o;
    uint32_t tsum = te, dsum = (valid && !is_out) ? (uint32_t)dwh : 0u;
    wave_all2<OpAdd, OpAdd>(tsum, dsum);
    const uint32_t Fe = FeBase + (tsum >> 1);
    const uint32_t Fc = is_out ? Fe : Fm + dP + (uint32_t)dwh;
    F[valid ? (is_out ? e : r) : N + 1] = Fc;
    const uint32_t Fn = valid ? Fc : 0u;
    const uint64_t S = start_of(cur, k) + (uint64_t)shift;
    uint32_t Dn = Fn, A, Bv;
    const uint32_t cnt = slo(valid, is_out ? kinde : (rq.z & 3u), is_out ? thre : rq.y, Pc, Fn, S, A, Bv);
    wave_all3<OpMax, OpMin, OpMax>(Dn, A, Bv);
    const uint32_t D0 = readlane(cur.D, k), cnt0 = readlane(cur.cnt, k), Fo = readlane(fo, k);
    // the scalar fields by v_writelane, the prefill (a vector register) by a select
    cand.Slo = wlane((uint32_t)S, k, cand.Slo);
    cand.Shi = wlane((uint32_t)(S >> 32), k, cand.Shi);
    cand.P = lane != k ? cand.P : Pc;
    cand.D = wlane(Dn, k, cand.D);
    cand.cnt = wlane(cnt, k, cand.cnt);
    cand.A = wlane(A, k, cand.A);
    cand.Bv = wlane(Bv, k, cand.Bv);
    dn += (int64_t)cnt - (int64_t)cnt0;
    const int64_t dSF = (int64_t)(bs - 1) * (int64_t)(int32_t)rfl(dP) + (int64_t)(int32_t)dsum + ((int64_t)rfl(Fe) - (int64_t)Fo);
    dt += (int64_t)bs * shift + dSF;
    return (int64_t)Dn - (int64_t)D0;
  }

  // Member recount of unchanged batch k whose start moved by `shift` out of its bounds.
  __device__ void recount_row(int k, int64_t shift, int64_t &dn) {
    const int q0 = k * B;
    const bool valid = lane < batch_size(k);
    const uint32_t r = valid ? (uint32_t)perm[min(q0 + lane, N - 1)] : (uint32_t)N;
    const uint4 rq = req[r];
    const uint32_t Fm = F[r];
    const uint64_t S = start_of(cur, k) + (uint64_t)shift;
    uint32_t A, Bv;
    const uint32_t cnt = slo(valid, rq.z & 3u, rq.y, readlane(cur.P, k), Fm, S, A, Bv);
    wave_all2<OpMin, OpMax>(A, Bv);
    cand.cnt = wlane(cnt, k, cand.cnt);
    cand.A = wlane(A, k, cand.A);
    cand.Bv = wlane(Bv, k, cand.Bv);
    dn += (int64_t)cnt - (int64_t)readlane(cur.cnt, k);
  }

  // Batches [k0, k1) keep their members and start `shift` later: new starts, latency
  // change, and the mask of those whose start leaves its bounds.
  __device__ uint64_t shift_range(int k0, int k1, int64_t shift, int64_t &dt) {
    const bool in = lane >= k0 && lane < k1;
    const uint64_t S = (((uint64_t)cur.Shi << 32) | cur.Slo) + (uint64_t)shift;
    cand.Slo = in ? (uint32_t)S : cand.Slo;
    cand.Shi = in ? (uint32_t)(S >> 32) : cand.Shi;
    const bool flip = in && (S > (uint64_t)cur.A || S < (uint64_t)cur.Bv);
    dt += shift * requests_in(k0, k1);
    return __ballot(flip);
  }

  __device__ void propose(const Move &mv, int64_t &dn, int64_t &dt, int &klast) {
    cand = cur;
    prologue(mv);
    dn = 0;
    dt = 0;
    int64_t carry = changed_row(mv.a, 0, dn, dt);
    const int64_t shift_mid = carry;  // start change of the batches between a and c (swap)
    uint64_t flagged = 0;
    if (mv.type == 2) {
      for (int k = mv.a + 1; k <= mv.c; ++k) carry += changed_row(k, carry, dn, dt);
    } else {
      // the batches strictly between a and c: candidate starts are written even for a
      // zero shift, since the records are copied on accept
      if (mv.c > mv.a + 1) flagged |= shift_range(mv.a + 1, mv.c, shift_mid, dt);
      carry += changed_row(mv.c, shift_mid, dn, dt);
    }
    const int kb = mv.c + 1;
    if (carry != 0 && kb < M) {
      flagged |= shift_range(kb, M, carry, dt);
      klast = M - 1;
    } else {
      klast = mv.c;
    }
    while (flagged) {
      const int k = __builtin_ctzll(flagged);
      flagged &= flagged - 1;
      recount_row(k, k >= kb ? carry : shift_mid, dn);
    }
  }

  // Restore F after a rejected proposal.
  __device__ void undo(const Move &mv) {
    for (int k = mv.a; k <= mv.c; ++k) {
      if (mv.type == 1 && k != mv.a && k != mv.c) continue;
      const int q0 = k * B;
      const bool valid = lane < batch_size(k);
      const uint4 t0 = tab[3 * k], t1 = tab[3 * k + 1];
      const uint32_t o = t0.x, Lo = t0.z, eo = t0.w, Le = t1.x, ee = t1.y, dP = t1.z;
      // as in changed_row: lanes past the batch read a clamped position, and they and the
      // leaving member write the spare slot F[n + 1] (no branch)
      const uint32_t r = valid ? (uint32_t)perm[min(q0 + lane, N - 1)] : (uint32_t)N;
      const uint32_t Lm = req[r].x >> 16;
      const uint32_t Fm = F[r];
      const uint32_t mue = min(Lm, Le), muo = min(Lm, Lo);
      const uint32_t wem = vmul24(mue, vmad24(d2, mue, ee));
      const uint32_t wom = vmul24(muo, vmad24(d2, muo, eo));
      const int32_t dwh = (int32_t)(wem - wom) >> 1;
      F[(valid && r != o) ? r : N + 1] = Fm - dP - (uint32_t)dwh;
    }
    // every leaving member's slot held a newcomer's candidate value
    if (lane < M && mv.changes(lane)) F[ovec] = fo;
    wave_sync_lds();
  }

  __device__ __forceinline__ void apply_move(int type, int i, int j) { apply_move_lds(perm, type, i, j, lane); }
};


// LDS of one chain of the one-batch-per-wave kernel: order, finish offsets (two spare
// slots), 48 bytes of proposal table per batch.
__host__ __device__ __forceinline__ size_t wave_chain_bytes(int n, int B) {
  const size_t M = (size_t)(n + B - 1) / B;
  return (((size_t)n * 2 + 15) & ~size_t(15)) + (((size_t)(n + 2) * 4 + 15) & ~size_t(15)) + M * 48;
}

// One chain by one wave: record slot `chain`, Philox chain index `rng_chain`, the request
// records in `req`, the chain's LDS at `wb`. OBJ: objective (0 attainment, then total
// latency; 1 ratio n / t).
template <int OBJ>
__device__ void anneal_wave_body(const DevModel &m, const StaticParams &sp, const uint4 *req, unsigned char *wb,
                                 int chains, int chain, uint32_t rng_chain, int iters, double T0, double alpha,
                                 uint32_t key0, uint32_t key1, uint64_t swap_thr, const SearchParams &srch,
                                 unsigned char *ws) {
  const int n = m.n, B = m.B;
  const int M = (n + B - 1) / B;
  const size_t perm_b = ((size_t)n * 2 + 15) & ~size_t(15);
  const size_t f_b = ((size_t)(n + 2) * 4 + 15) & ~size_t(15);
  const int lane = lane_id();
  WaveChain st;
  st.req = req;
  st.perm = reinterpret_cast<uint16_t *>(wb);
  st.F = reinterpret_cast<uint32_t *>(wb + perm_b);
  st.tab = reinterpret_cast<uint4 *>(wb + perm_b + f_b);
  st.d0 = sp.d0;
  st.d2 = sp.d2;
  st.N = n;
  st.B = B;
  st.M = M;
  st.lane = lane;
  st.fo = 0u;
  st.ovec = 0u;
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
      st.apply_move(mv.type, i, j);
    } else {
      int64_t dn, dt;
      int klast;
      st.propose(mv, dn, dt, klast);
      acc = obj_accept<OBJ>(cn, ct, dn, dt, t_ref, cool.T, w3);
      if (acc) {
        st.apply_move(mv.type, i, j);
        st.cur = st.cand;
        cn += dn;
        ct += (uint64_t)dt;
      } else {
        st.undo(mv);
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
template <int OBJ>
__global__ void __launch_bounds__(1024) anneal_wave_kernel(DevModel m, StaticParams sp, QueuePtrs q, int chains,
                                                            int iters, double T0, double alpha, uint32_t key0,
                                                            uint32_t key1, uint64_t swap_thr, SearchParams srch,
                                                            unsigned char *ws) {
  extern __shared__ __align__(16) unsigned char lds[];
  if (!gate_open(ws, m.gate, m.flags)) return;
  const int n = m.n;
  const int waves = blockDim.x >> 6;
  uint4 *req = reinterpret_cast<uint4 *>(lds);
  const int wave = uniform((int)(threadIdx.x >> 6));
  unsigned char *wb = lds + (size_t)(n + 1) * 16 + (size_t)wave * wave_chain_bytes(n, m.B);
  load_static_records(q, m, req);
  __syncthreads();
  const int chain = uniform((int)blockIdx.x * waves + wave);
  if (chain >= chains) return;
  anneal_wave_body<OBJ>(m, sp, req, wb, chains, chain, (uint32_t)chain, iters, T0, alpha, key0, key1, swap_thr, srch,
                        ws);
}

}  // namespace sa
