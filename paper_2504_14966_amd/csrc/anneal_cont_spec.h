// Continuous admission with two proposals scored per round (speculative pairs).
//
// Algorithm 1 scores one proposal at a time against the current order. Proposal k + 1 is
// scored against the same order whenever proposal k is rejected, so a round scores k and
// k + 1 against the current order at once: if k is accepted, the score of k + 1 is dropped
// and k + 1 is scored again in the next round against the new order; if k is rejected, the
// score of k + 1 is exactly the one the chain needs. The trajectory, accept count, digest
// and best order are those of scoring one proposal at a time, and a round completes two
// proposals whenever the first is rejected.
//
// One workgroup of two waves per chain: wave w scores proposal k + w. The replay is the
// list-scheduling one with 32-bit times (the running requests in a sliding window when at
// most 32 run, else one pop per step from lane 0), restarted at the chunk of admissions
// holding the candidate's first change; it is bound by the issue of its own serial steps,
// so the second wave of a chain works in issue slots the SIMD would otherwise leave empty.
// The waves meet once per round at the workgroup barrier, after which both take the same
// decisions from the two scores, and once more when a move is accepted (the first wave
// applies it to the shared records before either replays again).
//
// Candidate records are read from the current order's records through a branch-free
// position map, so one copy of them serves both waves. LDS per chain: those records
// (16 B per position, request id above the kind bits), per wave five 32-bit arrays of
// n + 1 entries (prefill prefix sums, run starts, run-end prefills, segment-cost prefix
// sums, TTFTs), three sets of admission pops plus chunk-start keys (the current
// order's and one per wave), and the two waves' scores in two slots used in alternate
// rounds. The request table is not staged in LDS: each chain reads its start order's
// records once from global memory.
#pragma once

#include "kernels.h"

namespace sa {

// Candidate position p reads current position src(p), without branches: position j reads
// i, and the positions in [rlo, rlo + rspan) read p + dir. An insert (remove at i,
// re-insert at j) shifts the positions between i and j by one towards i; a swap is the
// one-position range {i} reading j; the identity has no j and an empty range.
struct SrcMap {
  int j, ito, rlo, dir;
  uint32_t rspan;
  __device__ __forceinline__ int src(int p) const {
    const int shifted = (uint32_t)(p - rlo) < rspan ? p + dir : p;
    return p == j ? ito : shifted;
  }
};

__device__ __forceinline__ SrcMap src_map(int kind, int i, int j) {
  if (kind == 0 || i == j) return SrcMap{-1, 0, 0, 0, 0u};
  if (kind == 1) return SrcMap{j, i, i, j - i, 1u};
  if (i < j) return SrcMap{j, i, i, 1, (uint32_t)(j - i)};
  return SrcMap{j, i, j + 1, -1, (uint32_t)(i - j)};
}

// one wave's five arrays of n + 1 entries
__host__ __device__ __forceinline__ size_t spec_cand_bytes(int n) { return ((size_t)20 * (n + 1) + 15) / 16 * 16; }
// Admissions per chunk and running keys kept per chunk start: with at most 32 running, the
// sliding window's 64 - n0 admissions and 32 keys; with more, 64 admissions and n0 keys.
__host__ __device__ __forceinline__ int spec_chunk_len(int n0) { return n0 <= 32 ? 64 - n0 : 64; }
__host__ __device__ __forceinline__ int spec_snap_len(int n0) { return n0 <= 32 ? 32 : n0; }
// chunk-start keys of one order
__host__ __device__ __forceinline__ size_t spec_chunk_bytes(int n, int B) {
  const int n0 = n < B ? n : B, nadm = n - n0;
  const int S = spec_chunk_len(n0);
  return nadm > 0 ? (size_t)((nadm + S - 1) / S) * spec_snap_len(n0) * 4 : 0;
}
__host__ __device__ __forceinline__ size_t spec_pop_bytes(int n) { return ((size_t)4 * n + 15) / 16 * 16; }
// scores exchanged per round: 2 slots x 2 waves x 32 B
constexpr size_t kSpecXchBytes = 128;
// LDS of one chain (one workgroup)
__host__ __device__ __forceinline__ size_t spec_chain_bytes(int n, int B) {
  return kSpecXchBytes + (size_t)16 * n + 2 * spec_cand_bytes(n) + 3 * (spec_pop_bytes(n) + spec_chunk_bytes(n, B));
}

// The current order's admission state: pops, chunk-start keys (whose first n0 entries are
// the initial group's sorted keys whenever a request waits), the initial group's prefill
// and context sums; and the buffers of the two waves' candidates. Accepting candidate C
// swaps its buffers with the current ones. Both waves keep identical copies.
struct SpecCache {
  uint32_t *ev_cur, *snap_cur, *ev_c[2], *snap_c[2];
  uint32_t pr0_cur, c1_cur;
  template <int C>
  __device__ __forceinline__ void accept(uint32_t pr0, uint32_t c1) {
    uint32_t *t = ev_cur;
    ev_cur = ev_c[C];
    ev_c[C] = t;
    t = snap_cur;
    snap_cur = snap_c[C];
    snap_c[C] = t;
    pr0_cur = pr0;
    c1_cur = c1;
  }
};

// Score of one candidate of the current order. lo is the first position it changes:
// admissions before the window chunk holding it are the current order's. ev and snap
// receive the candidate's pops and chunk-start keys, sc holds its five arrays; pr0 and c1
// receive its initial group's sums. Every time fits 32 bits (checked on the device before
// the kernel runs).
__device__ __forceinline__ Score spec_replay(const DevModel &m, const uint4 *__restrict__ posr, const SrcMap sm,
                                             const int lo, const SpecCache &cc, uint32_t *ev, uint32_t *snap,
                                             uint32_t *sc, uint32_t &pr0, uint32_t &c1) {
  const int lane = lane_id();
  const int N = m.n, B = m.B;
  const int n0 = min(B, N), nadm = N - n0;
  const uint32_t d0 = (uint32_t)m.d0, d1 = (uint32_t)m.d1, d2 = (uint32_t)m.d2;
  const int W = N + 1;
  uint32_t *preA = sc, *rsA = sc + W, *runpre = sc + 2 * W, *segA = sc + 3 * W, *tta = sc + 4 * W;
  constexpr uint32_t kInf = 0xFFFFFFFFu;

  // initial group: positions 0 .. n0 - 1 start at step 0 (the current order's when the
  // candidate changes no position below n0)
  uint32_t list;
  if (lo >= n0) {
    list = lane < n0 ? cc.snap_cur[lane] : kInf;
    pr0 = cc.pr0_cur;
    c1 = cc.c1_cur;
  } else {
    uint32_t key = kInf, lin0 = 0, pf0 = 0;
    if (lane < n0) {
      const uint4 rq = posr[sm.src(lane)];
      key = ((rq.x >> 16) << 10) | (uint32_t)lane;
      lin0 = rq.x & 0xFFFFu;
      pf0 = rq.w;
    }
    pr0 = wsum32(pf0);
    c1 = wsum32(lin0);
    int rank = 0;
    for (int u = 0; u < n0; ++u) rank += rl(key, u) < key ? 1 : 0;
    if (lane < n0) runpre[rank] = key;
    wave_sync_lds();
    list = lane < n0 ? runpre[lane] : kInf;
    wave_sync_lds();
  }

  // admissions before the chunk holding the first changed one are the current order's
  const int Sfull = spec_chunk_len(n0), SN = spec_snap_len(n0);
  const int cr = lo >= n0 ? (lo - n0) / Sfull : 0;
  int done = min(cr * Sfull, nadm);
  for (int x = lane; x < done; x += kWave) ev[x] = cc.ev_cur[x];
  for (int x = lane; x < cr * SN; x += kWave) snap[x] = cc.snap_cur[x];
  if (done > 0) list = lane < n0 ? cc.snap_cur[cr * SN + lane] : kInf;
  if (n0 > 32) {
    // More than 32 running: the sorted keys fill lanes [0, n0), kInf above; a step pops
    // lane 0 and leaves lane i = max(list[i], min(list[i + 1], nk)); the pops enter lane 0
    // of a second register that moves up one lane per step.
    while (done < nadm) {
      const int cnt = min(kWave, nadm - done);
      if (lane < n0) snap[(done / kWave) * SN + lane] = list;
      uint32_t LP = 0;
      if (lane < cnt) {
        const int p = n0 + done + lane;
        LP = ((posr[sm.src(p)].x >> 16) << 10) | (uint32_t)p;
      }
      uint32_t evq = 0;
      uint32_t top = __builtin_amdgcn_readfirstlane(list);
      for (int t = 0; t < cnt; ++t) {
        const uint32_t nk = (top & ~1023u) + rl(LP, t);
        evq = dpp_old<kDppWaveShr1, 0xF>(list, evq);
        const uint32_t sh = dpp_old<kDppWaveShl1, 0xF>(kInf, list);
        list = max(list, min(sh, nk));
        top = __builtin_amdgcn_readfirstlane(list);
      }
      if (lane < cnt) ev[done + cnt - 1 - lane] = evq;
      done += cnt;
    }
  }
  // At most 32 running: a sliding window. Before step t of a chunk, lanes [0, t) hold the
  // keys popped so far and lanes [t, t + n0) the running keys, sorted, kInf above; popping
  // lane t and inserting key nk leaves lane i = median(list[i - 1], list[i], nk).
  while (done < nadm) {
    const int S = min(Sfull, nadm - done);
    if (lane < n0) snap[(done / Sfull) * 32 + lane] = list;
    uint32_t LP = 0;  // (l_out << 10) | position of the positions admitted in this chunk
    if (lane < S) {
      const int p = n0 + done + lane;
      LP = ((posr[sm.src(p)].x >> 16) << 10) | (uint32_t)p;
    }
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
  if (lane < n0) ev[nadm + lane] = list;
  if (lane == 0) preA[0] = 0u;
  wave_sync_lds();

  // pass A: segment costs, prefills, run starts and their prefix sums
  uint32_t fcarry = 0, Ccarry = c1, precarry = 0, rscarry = 0, segcarry = 0;
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
    const uint4 rq = posr[sm.src(v ? q : 0)];
    const uint4 ra = posr[sm.src(adm ? n0 + k - 1 : 0)];
    const uint32_t outq = v ? (rq.x & 0xFFFFu) + (rq.x >> 16) : 0u;
    const uint32_t la = adm ? (ra.x & 0xFFFFu) : 0u, pfa = adm ? ra.w : 0u;
    const uint32_t dC = v ? b * s - outq + la : 0u;  // two's complement: a signed change
    const uint32_t dCi = scan_add32(dC);
    const uint32_t Ck = Ccarry + dCi - dC;
    const uint32_t seg = s * (d0 + d1 * b + d2 * Ck) + (d2 * b) * ((s * (s + 1u)) >> 1);
    const uint32_t SEG = segcarry + scan_add32(seg);
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
    segcarry = rl(SEG, kWave - 1);
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
    const uint32_t SEG = v ? segA[kc] : 0u;
    const uint32_t e2e = pr0 + SEG + (rsk > 1 ? preA[max(rsk, 2u) - 1] : 0u);
    tta[(v && k <= nadm) ? k : 0] = pr0 + SEG + runpre[rsk];
    wave_sync_lds();
    const uint4 rq = posr[sm.src((int)q)];
    const uint32_t ttft = (int)q < n0 ? pr0 : tta[max((int)q - n0 + 1, 0)];
    const uint32_t kind = rq.z & 3u, thr = rq.y, L = rq.x >> 16;
    const bool met = v & (kind == 0 ? ttft <= thr
                                    : (kind == 2 ? e2e <= thr : (uint64_t)(e2e - ttft) <= (uint64_t)thr * L));
    tsum += v ? (uint64_t)e2e : 0ull;
    nmet += __popcll(__ballot(met));
  }
  wave_sync_lds();
  return Score{nmet, wave_sum_u64_dpp(tsum)};
}

// One workgroup of two waves per chain (blockDim 128, one chain per block).
template <int OBJ>
__global__ void __launch_bounds__(128) anneal_cont_spec_kernel(DevModel m, QueuePtrs q, int chains, int iters,
                                                                double T0, double alpha, uint32_t key0, uint32_t key1,
                                                                uint64_t swap_thr, SearchParams srch,
                                                                unsigned char *ws) {
  extern __shared__ __align__(16) unsigned char lds[];
  if (!gate_open(ws, m.gate, m.flags)) return;
  const int n = m.n;
  const int chain = (int)blockIdx.x;
  if (chain >= chains) return;
  const int w = uniform((int)(threadIdx.x >> 6));
  const int lane = lane_id();
  // scores of the two waves, slot r & 1 in round r: {n, t, pr0 | c1 << 32, unused}
  uint64_t *xch = reinterpret_cast<uint64_t *>(lds);
  uint4 *posr = reinterpret_cast<uint4 *>(lds + kSpecXchBytes);
  unsigned char *base = lds + kSpecXchBytes + (size_t)16 * n;
  uint32_t *sc = reinterpret_cast<uint32_t *>(base + (size_t)w * spec_cand_bytes(n));
  SpecCache cc{};
  {
    unsigned char *cb = base + 2 * spec_cand_bytes(n);
    const size_t evb = spec_pop_bytes(n), snb = spec_chunk_bytes(n, m.B);
    cc.ev_cur = reinterpret_cast<uint32_t *>(cb);
    cc.ev_c[0] = reinterpret_cast<uint32_t *>(cb + evb);
    cc.ev_c[1] = reinterpret_cast<uint32_t *>(cb + 2 * evb);
    cc.snap_cur = reinterpret_cast<uint32_t *>(cb + 3 * evb);
    cc.snap_c[0] = reinterpret_cast<uint32_t *>(cb + 3 * evb + snb);
    cc.snap_c[1] = reinterpret_cast<uint32_t *>(cb + 3 * evb + 2 * snb);
  }
  const WsHeader *h = reinterpret_cast<const WsHeader *>(ws);
  const int64_t t_ref = h->t_ref;
  int64_t cn = h->start_n;
  uint64_t ct = (uint64_t)h->start_t;
  const int64_t allmet = h->allmet;
  const uint16_t *start = reinterpret_cast<const uint16_t *>(ws + ws_off_start());
  const size_t stride = ws_perm_stride(n);
  uint16_t *gbest = reinterpret_cast<uint16_t *>(ws + ws_off_best(n, chains)) + (size_t)chain * stride;
  uint16_t *gcur = reinterpret_cast<uint16_t *>(ws + ws_off_cur(n, chains)) + (size_t)chain * stride;
  // the start order's records by position, with the request id above the kind bits
  for (int p = (int)threadIdx.x; p < n; p += 2 * kWave) {
    const uint16_t r = start[p];
    gbest[p] = r;
    const uint32_t lin = q.in_len[r], lout = q.out_len[r];
    posr[p] = make_uint4(lin | (lout << 16), q.thr[r], (uint32_t)q.kind[r] | ((uint32_t)r << 2),
                         (uint32_t)(m.p0 + m.p1 * lin));
  }
  __syncthreads();
  // the start order's state: each wave replays it into its own buffers, the first wave's
  // become the current ones (both waves compute the same sums)
  {
    uint32_t pr0, c1;
    spec_replay(m, posr, src_map(0, 0, 0), 0, cc, w ? cc.ev_c[1] : cc.ev_c[0], w ? cc.snap_c[1] : cc.snap_c[0], sc,
                pr0, c1);
    cc.accept<0>(pr0, c1);
  }
  __syncthreads();
  int64_t bn = cn;
  uint64_t bt = ct;
  int64_t biter = -1, accepts = 0;
  uint64_t digest = kFnvOffset;
  Cooling cool{T0, alpha, srch.level_len, srch.level_len};
  ProposalStream ps;  // iterations kb .. kb + 63
  int kb = 0, slot = 0;
  const int iters_run = (srch.early_exit && allmet) ? 0 : iters;
  if (iters_run > 0) ps.refill(0, lane, n, (uint32_t)chain, key0, key1, swap_thr, 0);
  for (int k = 0; k < iters_run;) {
    if (k + 1 - kb >= kWave) {
      kb = k;
      ps.refill(kb, lane, n, (uint32_t)chain, key0, key1, swap_thr, 0);
    }
    const bool two = k + 1 < iters_run;
    const uint32_t pk0 = rl(ps.pk, k - kb), pk1 = rl(ps.pk, k + 1 - kb);
    const int i0 = (int)(pk0 & 1023u), j0 = (int)((pk0 >> 10) & 1023u), t0 = (int)((pk0 >> 20) & 1u) + 1;
    const int i1 = (int)(pk1 & 1023u), j1 = (int)((pk1 >> 10) & 1023u), t1 = (int)((pk1 >> 20) & 1u) + 1;
    const int mi = w ? i1 : i0, mj = w ? j1 : j0, mt = w ? t1 : t0;
    uint32_t pr0, c1;
    // (the buffer pointers are selected, not indexed by the wave, which would place them in
    // scratch memory)
    uint32_t *my_ev = w ? cc.ev_c[1] : cc.ev_c[0], *my_snap = w ? cc.snap_c[1] : cc.snap_c[0];
    const Score s = spec_replay(m, posr, src_map(mt, mi, mj), min(mi, mj), cc, my_ev, my_snap, sc, pr0, c1);
    uint64_t *mine = xch + (slot * 2 + w) * 4;
    if (lane == 0) {
      mine[0] = (uint64_t)s.n;
      mine[1] = s.t;
      mine[2] = (uint64_t)pr0 | ((uint64_t)c1 << 32);
    }
    __syncthreads();
    const uint64_t *x0 = xch + (slot * 2) * 4, *x1 = xch + (slot * 2 + 1) * 4;
    const int64_t n0s = (int64_t)x0[0], n1s = (int64_t)x1[0];
    const uint64_t t0s = x0[1], t1s = x1[1], g0 = x0[2], g1 = x1[2];
    slot ^= 1;
    int kacc = -1, ai = 0, aj = 0, at = 0;
    if (obj_accept<OBJ>(cn, ct, n0s - cn, (int64_t)(t0s - ct), t_ref, cool.T, rl(ps.w3, k - kb))) {
      cool.step();
      cc.accept<0>((uint32_t)g0, (uint32_t)(g0 >> 32));
      kacc = k;
      ai = i0;
      aj = j0;
      at = t0;
      cn = n0s;
      ct = t0s;
      k += 1;
    } else {
      cool.step();
      if (two) {
        if (obj_accept<OBJ>(cn, ct, n1s - cn, (int64_t)(t1s - ct), t_ref, cool.T, rl(ps.w3, k + 1 - kb))) {
          cc.accept<1>((uint32_t)g1, (uint32_t)(g1 >> 32));
          kacc = k + 1;
          ai = i1;
          aj = j1;
          at = t1;
          cn = n1s;
          ct = t1s;
        }
        cool.step();
      }
      k += 2;
    }
    if (kacc >= 0) {
      ++accepts;
      digest = (digest ^ (uint64_t)kacc) * kFnvPrime;
      digest = (digest ^ (uint64_t)cn) * kFnvPrime;
      digest = (digest ^ ct) * kFnvPrime;
      const bool better = obj_better<OBJ>(cn, ct, bn, bt);
      if (better) {
        bn = cn;
        bt = ct;
        biter = kacc;
      }
      if (w == 0) {
        apply_move_lds(posr, ai == aj ? 0 : at, ai, aj, lane);
        if (better)
          for (int p = lane; p < n; p += kWave) gbest[p] = (uint16_t)(posr[p].z >> 2);
      }
      // both waves take this branch: the records change before either replays again
      __syncthreads();
    }
  }
  if (w == 0) {
    for (int p = lane; p < n; p += kWave) gcur[p] = (uint16_t)(posr[p].z >> 2);
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
}

}  // namespace sa
