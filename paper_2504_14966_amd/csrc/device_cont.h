// Continuous-admission timeline replay by one wave, lanes = batch slots (gfx950).
//
// Model (Background section of the paper: iteration-level scheduling; a prefill
// iteration stalls the running decodes): all requests are present at time 0; whenever a
// slot is free and requests wait, the next ones in priority order are admitted together
// with one prefill iteration costing the sum of their p0 + p1 * l_in; every decode
// iteration advances each running request by one token and costs d0 + d1 * b + d2 * ctx.
//
// Event form. Let K be the number of decode iterations so far and C the running
// requests' context sum before the next iteration. Admitting r at K adds l_in(r) to C and
// schedules its finish at K + l_out(r); finishing r at K removes l_in(r) + l_out(r); each
// iteration adds b to C. With the running set fixed, s iterations cost
//   s * (d0 + d1 * b + d2 * C) + d2 * b * s (s + 1) / 2,
// so the replay jumps from one finish step to the next (the minimum over the slots).
// Each slot keeps its request's TTFT; every SLO kind is judged when the request finishes
// (TPOT as e2e - TTFT <= thr * l_out). Cross-slot minima and sums are DPP row reductions
// plus v_readlane, so the clock, K, C and b stay in scalar registers; per-slot updates
// are selects rather than branches. Every event retires at least one request, so at most
// n events occur.
#pragma once
#include <type_traits>

#include "device_common.h"
#include "device_replay.h"

namespace sa {

template <int CTRL>
__device__ __forceinline__ uint32_t dpp_c(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, 0xF, 0xF, true);
}
__device__ __forceinline__ uint32_t rl(uint32_t v, int l) { return (uint32_t)__builtin_amdgcn_readlane((int)v, l); }

// wave-wide sum / min of 32-bit lane values (result uniform)
__device__ __forceinline__ uint32_t wsum32(uint32_t v) {
  v += dpp_c<0xB1>(v);
  v += dpp_c<0x4E>(v);
  v += dpp_c<0x141>(v);
  v += dpp_c<0x140>(v);
  return (rl(v, 0) + rl(v, 16)) + (rl(v, 32) + rl(v, 48));
}
__device__ __forceinline__ uint32_t wmin32(uint32_t v) {
  v = min(v, dpp_c<0xB1>(v));
  v = min(v, dpp_c<0x4E>(v));
  v = min(v, dpp_c<0x141>(v));
  v = min(v, dpp_c<0x140>(v));
  return min(min(rl(v, 0), rl(v, 16)), min(rl(v, 32), rl(v, 48)));
}

constexpr uint32_t kIdle = 0xFFFFFFFFu;

// req record: x = l_in | l_out << 16, y = threshold, z = kind (low 2 bits), w = prefill cost.
// The host guarantees (DevModel flags bit 1) that group prefill sums, d0 + d1 b + d2 C and
// d2 b fit 32 bits, so each event's cost is two 32 x 32 -> 64-bit products.
template <bool DETAIL>
__device__ Score replay_cont_fast(const DevModel &m, const uint4 *__restrict__ req, const uint16_t *perm, Remap rm,
                                  int64_t *detail) {
  const int lane = lane_id();
  const int N = m.n, B = m.B;
  const uint32_t d0 = (uint32_t)m.d0, d1 = (uint32_t)m.d1, d2 = (uint32_t)m.d2;
  uint32_t fK = kIdle, L = 0, thr = 0, kind = 0, lpl = 0;
  uint64_t ttft = 0;
  int r = 0;
  uint32_t K = 0, C = 0;
  uint64_t clock = 0, tsum = 0;
  int next = 0, b = 0;
  int64_t nmet = 0;
  for (int ev = 0; ev <= N; ++ev) {
    const int g = (next < N && b < B) ? min(B - b, N - next) : 0;
    if (g > 0) {
      const bool freel = lane < B && fK == kIdle;
      const int rank = rank_in_mask(__ballot(freel));
      const bool adm = freel && rank < g;
      const int rr = perm[rm.src(min(next + rank, N - 1))];
      const uint4 rq = req[rr];
      const uint32_t lin = adm ? (rq.x & 0xFFFFu) : 0u;
      const uint32_t pf = adm ? rq.w : 0u;
      const uint32_t Lr = rq.x >> 16;
      clock += wsum32(pf);
      C += wsum32(lin);
      r = adm ? rr : r;
      L = adm ? Lr : L;
      thr = adm ? rq.y : thr;
      kind = adm ? (rq.z & 3u) : kind;
      lpl = adm ? lin + Lr : lpl;
      fK = adm ? K + Lr : fK;
      ttft = adm ? clock : ttft;
      b += g;
      next += g;
    }
    const uint32_t fmin = wmin32(fK);
    const uint32_t s = fmin - K;
    const uint32_t X = d0 + d1 * (uint32_t)b + d2 * C;
    clock += (uint64_t)s * X + (uint64_t)(d2 * (uint32_t)b) * ((s * (s + 1u)) >> 1);
    C += (uint32_t)b * s;
    K = fmin;
    const bool fin = fK == K;
    const bool met = kind == 0 ? ttft <= (uint64_t)thr
                               : (kind == 2 ? clock <= (uint64_t)thr : clock - ttft <= (uint64_t)thr * L);
    if (DETAIL && fin) {
      detail[2 * r] = (int64_t)ttft;
      detail[2 * r + 1] = (int64_t)clock;
    }
    const uint64_t finm = __ballot(fin);
    const int nf = __popcll(finm);
    nmet += __popcll(__ballot(fin && met));
    tsum += clock * (uint32_t)nf;
    C -= nf == 1 ? rl(lpl, __builtin_ctzll(finm)) : wsum32(fin ? lpl : 0u);
    fK = fin ? kIdle : fK;
    b -= nf;
    if (b == 0 && next >= N) break;
  }
  return Score{nmet, tsum};
}

}  // namespace sa

namespace sa {

// ---------------------------------------------------------------------------------------
// Continuous admission in O(n) wave operations: list scheduling, then scans.
//
// In decode-step units continuous batching is list scheduling on B identical slots: the
// first min(B, n) requests start at step 0, and every time a running request finishes (the
// smallest finish step among the running ones) the next request in priority order takes
// its slot at that step and finishes l_out steps later. So the k-th finish event (in step
// order) is the k-th pop of a sorted list of the running requests' finish steps, and event
// k admits position min(B, n) + k - 1 while requests wait. The list lives in lanes,
// ascending: a pop is a one-lane DPP wave shift and an insert is a ballot plus a select.
// Keys pack (finish step << 10 | position), so ties are broken by position; which of two
// requests finishing at the same step is popped first changes no result.
//
// The clock then follows from prefix sums over the events. Between events k-1 and k
// (s_k = f_k - f_{k-1} decode steps) the running count is b_k = min(n0, n - k + 1), and the
// context sum C_k at the segment start obeys C_{k+1} = C_k + b_k s_k - (l + l_out of the
// finishing request) + (l of the admitted request). The segment costs
//   seg_k = s_k (d0 + d1 b_k + d2 C_k) + d2 b_k s_k (s_k + 1) / 2,
// and event k's admission adds its prefill pre_k. All finishes at one step happen before
// that step's single admission group, so with SEG and PRE the inclusive prefix sums and
// [rs_k, re_k] the run of events sharing step f_k:
//   e2e(finishing request of k) = PR0 + SEG_k + PRE_{rs_k - 1},
//   TTFT(request admitted at k) = PR0 + SEG_k + PRE_{re_k},
// where PR0 is the prefill of the initial group. Scans are DPP row shifts plus row
// broadcasts (6 steps for 64 lanes).
// ---------------------------------------------------------------------------------------

constexpr int kDppRowShr1 = 0x111, kDppRowShr2 = 0x112, kDppRowShr4 = 0x114, kDppRowShr8 = 0x118;
constexpr int kDppRowBcast15 = 0x142, kDppRowBcast31 = 0x143, kDppWaveShl1 = 0x130, kDppWaveShr1 = 0x138;

template <int CTRL, int ROWMASK>
__device__ __forceinline__ uint32_t dpp_old(uint32_t old, uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)old, (int)v, CTRL, ROWMASK, 0xF, false);
}

// v in the lanes of mask, 0 elsewhere, as one v_cndmask (a select the compiler cannot turn
// into a branch around the instruction that produced v)
__device__ __forceinline__ uint32_t keep_lanes(uint32_t v, uint64_t mask) {
  uint32_t r;
  asm("v_cndmask_b32_e64 %0, 0, %1, %2" : "=v"(r) : "v"(v), "s"(mask));
  return r;
}

__device__ __forceinline__ uint32_t add_sat(uint32_t a, uint32_t b) { return __builtin_elementwise_add_sat(a, b); }

// Inclusive scan over the 64 lanes with additions that saturate at 2^32 - 1: every value is
// nonnegative, so each lane gets min(its true prefix sum, 2^32 - 1) whatever the order.
__device__ __forceinline__ uint32_t scan_add_sat32(uint32_t v) {
  v = add_sat(v, dpp_old<kDppRowShr1, 0xF>(0u, v));
  v = add_sat(v, dpp_old<kDppRowShr2, 0xF>(0u, v));
  v = add_sat(v, dpp_old<kDppRowShr4, 0xF>(0u, v));
  v = add_sat(v, dpp_old<kDppRowShr8, 0xF>(0u, v));
  v = add_sat(v, dpp_old<kDppRowBcast15, 0xA>(0u, v));
  v = add_sat(v, dpp_old<kDppRowBcast31, 0xC>(0u, v));
  return v;
}

// Maximum of v over the lane's batch [b0, b1], exact at the batch's last lane b1: a max-scan
// confined to batches. Every DPP step runs on the whole wave (a lane left out would read as 0
// to its neighbour): in the row shifts the sending lane zeroes its value unless its batch
// reaches the receiver; in the row broadcasts (one sender, many receivers) the receiver keeps
// the value only when its batch starts at or below the sending lane (15 or 47, then 31).
__device__ __forceinline__ uint32_t seg_max32(uint32_t v, int b0, int b1, int lane) {
  v = max(v, dpp_old<kDppRowShr1, 0xF>(0u, b1 >= lane + 1 ? v : 0u));
  v = max(v, dpp_old<kDppRowShr2, 0xF>(0u, b1 >= lane + 2 ? v : 0u));
  v = max(v, dpp_old<kDppRowShr4, 0xF>(0u, b1 >= lane + 4 ? v : 0u));
  v = max(v, dpp_old<kDppRowShr8, 0xF>(0u, b1 >= lane + 8 ? v : 0u));
  v = max(v, keep_lanes(dpp_old<kDppRowBcast15, 0xA>(0u, v), __ballot(b0 <= (lane | 15) - 16)));
  v = max(v, keep_lanes(dpp_old<kDppRowBcast31, 0xC>(0u, v), __ballot(b0 <= 31)));
  return v;
}

// inclusive scans over the 64 lanes
__device__ __forceinline__ uint32_t scan_add32(uint32_t v) {
  v += dpp_old<kDppRowShr1, 0xF>(0u, v);
  v += dpp_old<kDppRowShr2, 0xF>(0u, v);
  v += dpp_old<kDppRowShr4, 0xF>(0u, v);
  v += dpp_old<kDppRowShr8, 0xF>(0u, v);
  v += dpp_old<kDppRowBcast15, 0xA>(0u, v);
  v += dpp_old<kDppRowBcast31, 0xC>(0u, v);
  return v;
}
__device__ __forceinline__ uint32_t scan_max32(uint32_t v) {
  v = max(v, dpp_old<kDppRowShr1, 0xF>(0u, v));
  v = max(v, dpp_old<kDppRowShr2, 0xF>(0u, v));
  v = max(v, dpp_old<kDppRowShr4, 0xF>(0u, v));
  v = max(v, dpp_old<kDppRowShr8, 0xF>(0u, v));
  v = max(v, dpp_old<kDppRowBcast15, 0xA>(0u, v));
  v = max(v, dpp_old<kDppRowBcast31, 0xC>(0u, v));
  return v;
}
// one step of four interleaved inclusive add-scans
template <int CTRL, int ROWMASK>
__device__ __forceinline__ void scan_step4(uint32_t &a, uint32_t &b, uint32_t &c, uint32_t &d) {
  a += dpp_old<CTRL, ROWMASK>(0u, a);
  b += dpp_old<CTRL, ROWMASK>(0u, b);
  c += dpp_old<CTRL, ROWMASK>(0u, c);
  d += dpp_old<CTRL, ROWMASK>(0u, d);
}
// Sum of 64-bit values over the 64 lanes (mod 2^64), exactly, as four 16-bit limb sums
// (each below 2^22) scanned together by DPP: no round trip through the LDS unit.
__device__ __forceinline__ uint64_t wave_sum_u64_dpp(uint64_t v) {
  uint32_t a0 = (uint32_t)v & 0xFFFFu, a1 = (uint32_t)v >> 16, a2 = (uint32_t)(v >> 32) & 0xFFFFu;
  uint32_t a3 = (uint32_t)(v >> 48);
  scan_step4<kDppRowShr1, 0xF>(a0, a1, a2, a3);
  scan_step4<kDppRowShr2, 0xF>(a0, a1, a2, a3);
  scan_step4<kDppRowShr4, 0xF>(a0, a1, a2, a3);
  scan_step4<kDppRowShr8, 0xF>(a0, a1, a2, a3);
  scan_step4<kDppRowBcast15, 0xA>(a0, a1, a2, a3);
  scan_step4<kDppRowBcast31, 0xC>(a0, a1, a2, a3);
  return (uint64_t)rl(a0, kWave - 1) + ((uint64_t)rl(a1, kWave - 1) << 16) + ((uint64_t)rl(a2, kWave - 1) << 32) +
         ((uint64_t)rl(a3, kWave - 1) << 48);
}

template <int CTRL, int ROWMASK>
__device__ __forceinline__ uint64_t add_dpp64(uint64_t v) {
  const uint32_t lo = dpp_old<CTRL, ROWMASK>(0u, (uint32_t)v), hi = dpp_old<CTRL, ROWMASK>(0u, (uint32_t)(v >> 32));
  return v + (((uint64_t)hi << 32) | lo);
}
__device__ __forceinline__ uint64_t scan_add64(uint64_t v) {
  v = add_dpp64<kDppRowShr1, 0xF>(v);
  v = add_dpp64<kDppRowShr2, 0xF>(v);
  v = add_dpp64<kDppRowShr4, 0xF>(v);
  v = add_dpp64<kDppRowShr8, 0xF>(v);
  v = add_dpp64<kDppRowBcast15, 0xA>(v);
  v = add_dpp64<kDppRowBcast31, 0xC>(v);
  return v;
}
// 64-bit inclusive max-scan over the 64 lanes.
__device__ __forceinline__ uint64_t scan_max64_step(uint64_t v, uint32_t lo, uint32_t hi) {
  const uint64_t o = ((uint64_t)hi << 32) | lo;
  return o > v ? o : v;
}
template <int CTRL, int ROWMASK>
__device__ __forceinline__ uint64_t max_dpp64(uint64_t v) {
  return scan_max64_step(v, dpp_old<CTRL, ROWMASK>(0u, (uint32_t)v), dpp_old<CTRL, ROWMASK>(0u, (uint32_t)(v >> 32)));
}
__device__ __forceinline__ uint64_t scan_max64(uint64_t v) {
  v = max_dpp64<kDppRowShr1, 0xF>(v);
  v = max_dpp64<kDppRowShr2, 0xF>(v);
  v = max_dpp64<kDppRowShr4, 0xF>(v);
  v = max_dpp64<kDppRowShr8, 0xF>(v);
  v = max_dpp64<kDppRowBcast15, 0xA>(v);
  v = max_dpp64<kDppRowBcast31, 0xC>(v);
  return v;
}

__device__ __forceinline__ uint64_t rl64(uint64_t v, int l) {
  return ((uint64_t)rl((uint32_t)(v >> 32), l) << 32) | rl((uint32_t)v, l);
}

// median of three unsigned values (c wave-uniform)
__device__ __forceinline__ uint32_t med3_u32(uint32_t a, uint32_t b, uint32_t c) {
  uint32_t d;
  asm("v_med3_u32 %0, %1, %2, %3" : "=v"(d) : "v"(a), "v"(b), "s"(c));
  return d;
}

// Per-wave LDS scratch of the list-scheduling replay (bytes, 16-aligned): event keys,
// prefill prefix sums, run starts, run-end prefills (4 B per event), segment-cost prefix
// sums and TTFTs (8 B per event), and the candidate order's request records by position.
__host__ __device__ __forceinline__ size_t cont_ls_off_seg(int n) { return ((size_t)4 * n + 12 * (size_t)(n + 1) + 7) / 8 * 8; }
__host__ __device__ __forceinline__ size_t cont_ls_off_pos(int n) { return (cont_ls_off_seg(n) + 16 * (size_t)(n + 1) + 15) / 16 * 16; }
__host__ __device__ __forceinline__ size_t cont_ls_scratch_bytes(int n) { return cont_ls_off_pos(n) + 16 * (size_t)n; }

// Kept by the annealing kernel between proposals when min(B, n) <= 32 (sliding window):
// the current order's admission pops, the running keys at the start of every window chunk
// and its initial group, plus the same for the candidate. A candidate that changes only
// positions >= lo keeps the current order's first admissions, so its replay restarts at
// the window chunk holding admission lo - n0 from that chunk's running keys.
struct LsCache {
  // with a cache the records by position (in the scratch) are the candidate order's: the
  // kernel applies each move to them and takes it back on reject
  uint32_t *ev_cur, *ev_cand;      // n pops each
  uint32_t *snap_cur, *snap_cand;  // running keys at the start of chunk c, at [32 c + lane]
  uint32_t list0_cur, list0_cand;  // initial group's sorted keys (lanes < n0), kInf above
  uint32_t pr0_cur, pr0_cand;      // its prefill sum
  uint32_t c1_cur, c1_cand;        // its context sum
  int lo;                          // first position the candidate changes
  __device__ __forceinline__ void accept() {
    uint32_t *t = ev_cur;
    ev_cur = ev_cand;
    ev_cand = t;
    t = snap_cur;
    snap_cur = snap_cand;
    snap_cand = t;
    list0_cur = list0_cand;
    pr0_cur = pr0_cand;
    c1_cur = c1_cand;
  }
};
// LDS for one LsCache: two pop arrays and two snapshot arrays
__host__ __device__ __forceinline__ size_t cont_inc_bytes(int n, int B) {
  const int n0 = n < B ? n : B, nadm = n - n0;
  const size_t chunks = nadm > 0 ? (size_t)((nadm + (64 - n0) - 1) / (64 - n0)) : 0;
  return 2 * (((size_t)4 * n + 15) / 16 * 16) + 2 * chunks * 32 * 4;
}

__device__ __forceinline__ uint32_t scan_add(uint32_t v) { return scan_add32(v); }
__device__ __forceinline__ uint64_t scan_add(uint64_t v) { return scan_add64(v); }
__device__ __forceinline__ uint32_t rl_any(uint32_t v, int l) { return rl(v, l); }
__device__ __forceinline__ uint64_t rl_any(uint64_t v, int l) { return rl64(v, l); }

// NARROW: every time on the timeline fits 32 bits (the device check bounds the total by
// sum(prefill) + (d0 + d1) sum(l_out) + d2 sum(l_out l_in + l_out (l_out + 1) / 2)).
template <bool DETAIL, bool NARROW, bool INC = false>
__device__ Score replay_cont_ls(const DevModel &m, const uint4 *__restrict__ req, const uint16_t *perm, Remap rm,
                                unsigned char *scratch, int64_t *detail, LsCache *cache = nullptr) {
  using TT = typename std::conditional<NARROW, uint32_t, uint64_t>::type;
  const int lane = lane_id();
  const int N = m.n, B = m.B;
  const int n0 = min(B, N), nadm = N - n0;
  const uint32_t d0 = (uint32_t)m.d0, d1 = (uint32_t)m.d1, d2 = (uint32_t)m.d2;
  uint32_t *ev = INC ? cache->ev_cand : reinterpret_cast<uint32_t *>(scratch);  // key of event k at [k - 1]
  uint32_t *preA = reinterpret_cast<uint32_t *>(scratch) + N;  // PRE_k at [k], PRE_0 = 0
  uint32_t *rsA = preA + (N + 1);                         // run start of event k at [k]
  uint32_t *runpre = rsA + (N + 1);                       // PRE at the end of the run starting at k
  TT *segA = reinterpret_cast<TT *>(scratch + cont_ls_off_seg(N));
  TT *tta = segA + (N + 1);                               // TTFT of the request admitted at event k
  uint4 *posr = reinterpret_cast<uint4 *>(scratch + cont_ls_off_pos(N));  // record of the request at position p
  constexpr uint32_t kInf = 0xFFFFFFFFu;

  // the candidate order's records, so later lookups by position are one LDS read (kept by
  // the annealing kernel, which applies each move to them, when a cache is given)
  if (!INC) {
    for (int p = lane; p < N; p += kWave) posr[p] = req[perm[rm.src(p)]];
    wave_sync_lds();
  }

  // initial group: positions 0 .. n0-1 start at step 0 (kept from the current order when
  // the candidate changes no position below n0)
  uint32_t list, pr0u, C1;
  if (INC && cache->lo >= n0) {
    list = cache->list0_cur;
    pr0u = cache->pr0_cur;
    C1 = cache->c1_cur;
  } else {
    uint32_t key = kInf, lin0 = 0, pf0 = 0;
    if (lane < n0) {
      const uint4 rq = posr[lane];
      key = ((rq.x >> 16) << 10) | (uint32_t)lane;
      lin0 = rq.x & 0xFFFFu;
      pf0 = rq.w;
    }
    pr0u = wsum32(pf0);
    C1 = wsum32(lin0);
    int rank = 0;
    for (int u = 0; u < n0; ++u) rank += rl(key, u) < key ? 1 : 0;
    if (lane < n0) runpre[rank] = key;
    wave_sync_lds();
    list = lane < n0 ? runpre[lane] : kInf;
    wave_sync_lds();
  }
  if (INC) {
    cache->list0_cand = list;
    cache->pr0_cand = pr0u;
    cache->c1_cand = C1;
  }
  const TT PR0 = (TT)pr0u;

  // list scheduling: pop the earliest finish, admit the next position at that step.
  if (n0 <= 32) {
    // Sliding window: before step t of a chunk lanes [0, t) hold the keys popped so far
    // and lanes [t, t + n0) the running keys, sorted, with kInf above. Popping list[t] and
    // inserting nk leaves lane i = median(list[i - 1], list[i], nk) for every lane: below
    // t the medians return the pops unchanged (they are sorted and below nk), at t the pop
    // itself, above t the merge of the remaining keys with nk. After S = 64 - n0 steps
    // the pops are stored and the window moves back to lane 0.
    const int Sfull = kWave - n0;
    int done = 0;
    if (INC) {
      // the candidate's admissions before the chunk holding its first change are the
      // current order's: copy their pops and chunk-start keys, restart from that chunk
      const int cr = cache->lo >= n0 ? (cache->lo - n0) / Sfull : 0;
      done = min(cr * Sfull, nadm);
      for (int x = lane; x < done; x += kWave) cache->ev_cand[x] = cache->ev_cur[x];
      for (int x = lane; x < cr * 32; x += kWave) cache->snap_cand[x] = cache->snap_cur[x];
      if (done > 0) list = lane < n0 ? cache->snap_cur[cr * 32 + lane] : kInf;
    }
    while (done < nadm) {
      const int S = min(Sfull, nadm - done);
      if (INC && lane < n0) cache->snap_cand[(done / Sfull) * 32 + lane] = list;
      uint32_t LP = 0;  // (l_out << 10) | position of the positions admitted in this chunk
      if (lane < S) {
        const int p = n0 + done + lane;
        LP = ((posr[p].x >> 16) << 10) | (uint32_t)p;
      }
      // Step t pops lane t and admits the key (f_t << 10) + LP[t], formed in lane t by the
      // vector unit and read out once: the step's dependence chain is the median, two
      // vector operations and one lane read. Unrolled by hand (the lane operations are
      // convergent, which keeps the compiler from unrolling a loop of run-time length).
      auto step = [&](int t) {
        const uint32_t nk = rl((list & ~1023u) + LP, t);
        const uint32_t below = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)list, kDppWaveShr1, 0xF, 0xF, true);
        list = med3_u32(below, list, nk);
      };
      int t = 0;
      for (; t + 4 <= S; t += 4) {
        step(t);
        step(t + 1);
        step(t + 2);
        step(t + 3);
      }
      for (; t < S; ++t) step(t);
      if (lane < S) ev[done + lane] = list;
      const uint32_t moved = (uint32_t)__builtin_amdgcn_ds_bpermute((lane + S) << 2, (int)list);
      list = lane < n0 ? moved : kInf;
      done += S;
    }
  } else {
    // With the list sorted, lane i of the list after the pop and the insert of nk is the
    // median of list[i], list[i + 1] and nk, i.e. max(list[i], min(list[i + 1], nk)). The
    // popped keys enter lane 0 of a second register that moves up one lane per step, so
    // after a chunk of cnt steps lane cnt - 1 - t holds the pop of step t.
    for (int c0 = 0; c0 < nadm; c0 += kWave) {
      const int cnt = min(kWave, nadm - c0);
      uint32_t LP = 0;
      if (lane < cnt) {
        const int p = n0 + c0 + lane;
        LP = ((posr[p].x >> 16) << 10) | (uint32_t)p;
      }
      uint32_t evq = 0;
      uint32_t top = __builtin_amdgcn_readfirstlane(list);
      for (int t = 0; t < cnt; ++t) {
        const uint32_t nk = (top & ~1023u) + rl(LP, t);
        evq = dpp_old<kDppWaveShr1, 0xF>(list, evq);  // lane 0 takes list[0], the key popped now
        const uint32_t sh = dpp_old<kDppWaveShl1, 0xF>(kInf, list);
        list = max(list, min(sh, nk));
        top = __builtin_amdgcn_readfirstlane(list);
      }
      if (lane < cnt) ev[c0 + cnt - 1 - lane] = evq;
    }
  }
  if (lane < n0) ev[nadm + lane] = list;
  if (lane == 0) preA[0] = 0u;
  wave_sync_lds();

  // pass A: segment costs, prefills, run starts and their prefix sums
  uint32_t fcarry = 0, Ccarry = C1, precarry = 0, rscarry = 0;
  TT segcarry = 0;
  for (int c0 = 0; c0 < N; c0 += kWave) {
    const int k = c0 + lane + 1;
    const bool v = k <= N;
    const uint32_t kk = v ? ev[k - 1] : 0u;
    const uint32_t f = kk >> 10;
    const int q = (int)(kk & 1023u);
    const uint32_t fprev = dpp_old<kDppWaveShr1, 0xF>(fcarry, f);
    const uint32_t s = v ? f - fprev : 0u;
    const uint32_t b = (uint32_t)min(n0, N - k + 1);
    const bool adm = v && k <= nadm;
    const uint4 rq = posr[v ? q : 0];
    const uint4 ra = posr[adm ? n0 + k - 1 : 0];
    const uint32_t outq = v ? (rq.x & 0xFFFFu) + (rq.x >> 16) : 0u;
    const uint32_t la = adm ? (ra.x & 0xFFFFu) : 0u, pfa = adm ? ra.w : 0u;
    const uint32_t dC = v ? b * s - outq + la : 0u;  // two's complement: a signed change
    const uint32_t dCi = scan_add32(dC);
    const uint32_t Ck = Ccarry + dCi - dC;
    // (lanes past the events, none when 64 divides n, have s = 0 and so seg = 0; they read
    // clamped positions and store to entry 0 of each array, which no read uses, so that the
    // passes have no branches)
    const TT seg = (TT)s * (TT)(d0 + d1 * b + d2 * Ck) + (TT)(d2 * b) * (TT)((s * (s + 1u)) >> 1);
    const TT SEG = segcarry + scan_add(seg);
    const uint32_t PRE = precarry + scan_add32(pfa);
    const uint32_t rs = max(rscarry, scan_max32((v && (k == 1 || s != 0)) ? (uint32_t)k : 0u));
    const uint32_t fnext = k < N ? (ev[min(k, N - 1)] >> 10) : kInf;
    const int kw = v ? k : 0;
    preA[kw] = PRE;
    rsA[kw] = rs;
    segA[kw] = SEG;
    runpre[(v && (k == N || fnext != f)) ? rs : 0u] = PRE;
    fcarry = rl(f, kWave - 1);
    Ccarry += rl(dCi, kWave - 1);
    segcarry = rl_any(SEG, kWave - 1);
    precarry = rl(PRE, kWave - 1);
    rscarry = rl(rs, kWave - 1);
  }
  wave_sync_lds();

  // pass B: end-to-end latency of each finishing request, TTFT of each admitted one, SLOs
  uint64_t tsum = 0;
  int64_t nmet = 0;
  for (int c0 = 0; c0 < N; c0 += kWave) {
    const int k = c0 + lane + 1;
    const bool v = k <= N;
    const int kc = min(k, N);
    const uint32_t q = v ? (ev[kc - 1] & 1023u) : 0u, rsk = v ? rsA[kc] : 1u;
    const TT SEG = v ? segA[kc] : (TT)0;
    const TT e2e = PR0 + SEG + (TT)(rsk > 1 ? preA[max(rsk, 2u) - 1] : 0u);
    tta[(v && k <= nadm) ? k : 0] = PR0 + SEG + (TT)runpre[rsk];
    wave_sync_lds();
    const uint4 rq = posr[q];
    const TT ttft = (int)q < n0 ? PR0 : tta[max((int)q - n0 + 1, 0)];
    const uint32_t kind = rq.z & 3u, thr = rq.y, L = rq.x >> 16;
    const bool met = v & (kind == 0 ? ttft <= (TT)thr
                                    : (kind == 2 ? e2e <= (TT)thr : (uint64_t)(e2e - ttft) <= (uint64_t)thr * L));
    tsum += v ? (uint64_t)e2e : 0ull;
    if (DETAIL && v) {
      const int r = perm[rm.src((int)q)];
      detail[2 * r] = (int64_t)ttft;
      detail[2 * r + 1] = (int64_t)e2e;
    }
    nmet += __popcll(__ballot(met));
  }
  wave_sync_lds();
  return Score{nmet, wave_sum_u64_dpp(tsum)};
}

}  // namespace sa
