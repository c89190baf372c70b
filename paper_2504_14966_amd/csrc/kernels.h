// Kernels of the annealing hot path (gfx950, wave64).
//
//   eval_kernel    : one wave per priority order; validates the row, replays it.
//   start_kernel   : Algorithm 1 initialisation (one workgroup): solo latency of every
//                    request, stable bitonic sort by (solo, id), scores of the sorted and
//                    the input orders, t_ref; writes the workspace header and start order.
//   anneal_kernel  : one wave per chain; per iteration a Philox block, a candidate order
//                    built on the fly from the current one, its replay, the Metropolis
//                    test and best-so-far tracking.
//   reduce_kernel  : lexicographic argmax over chains (n desc, t asc, chain asc).
//   small copy kernels for the readouts and the Fisher-Yates family.
#pragma once
#include "device_common.h"
#include "device_plan.h"
#include "device_replay.h"
#include "device_rng.h"
#include "device_cont.h"

namespace sa {

constexpr int kWavesPerBlock = 4;
constexpr int kBlock = kWave * kWavesPerBlock;

// Cooperative, coalesced load of the request records into LDS.
__device__ __forceinline__ void load_requests(const QueuePtrs &q, const DevModel &m, uint4 *req) {
  for (int r = threadIdx.x; r < m.n; r += blockDim.x) {
    const uint32_t lin = q.in_len[r], lout = q.out_len[r];
    req[r] = make_uint4(lin | (lout << 16), q.thr[r], (uint32_t)q.kind[r], (uint32_t)(m.p0 + m.p1 * lin));
  }
}

// Replay of one order: static closed form, or the continuous event loop (32-bit prefill
// sums when they fit, the 64-bit variant otherwise).
template <bool DETAIL>
__device__ __forceinline__ Score replay_any(const DevModel &m, const uint4 *req, const uint16_t *perm, Remap rm,
                                            uint4 *stage, int64_t *detail) {
  if (m.policy != 1) return replay_static<DETAIL>(m, req, perm, rm, stage, detail);  // both static policies
  if (m.flags & kFlagNarrowPrefill) return replay_cont_fast<DETAIL>(m, req, perm, rm, detail);
  return replay_continuous<DETAIL>(m, req, perm, rm, detail);
}

__device__ __forceinline__ size_t lds_align(size_t x) { return (x + 15) & ~size_t(15); }

template <bool DETAIL>
__global__ void __launch_bounds__(kBlock) eval_kernel(DevModel m, QueuePtrs q, const uint16_t *__restrict__ perms,
                                                       int64_t rows, int64_t *__restrict__ out,
                                                       int64_t *__restrict__ detail) {
  extern __shared__ __align__(16) unsigned char lds[];
  const EvalRows span = eval_gate(q, m, rows, out);
  if (span.end <= span.begin) return;
  const int n = m.n;
  uint4 *req = reinterpret_cast<uint4 *>(lds);
  const bool ls = m.policy == 1 && (m.flags & kFlagListSched);
  // continuous admission always leaves room for the list-scheduling scratch (the host sizes
  // the LDS by the policy; whether the list scheduling runs is the device check's)
  const size_t per_wave =
      lds_align((size_t)n * 2) + 64 * 16 + 32 * 4 + (m.policy == 1 ? lds_align(cont_ls_scratch_bytes(n)) : 0);
  const int wave = uniform((int)(threadIdx.x >> 6));
  unsigned char *wbase = lds + lds_align((size_t)n * 16) + (size_t)wave * per_wave;
  uint16_t *perm = reinterpret_cast<uint16_t *>(wbase);
  uint4 *stage = reinterpret_cast<uint4 *>(wbase + lds_align((size_t)n * 2));
  uint32_t *bitmap = reinterpret_cast<uint32_t *>(wbase + lds_align((size_t)n * 2) + 64 * 16);
  unsigned char *scratch = wbase + lds_align((size_t)n * 2) + 64 * 16 + 32 * 4;
  load_requests(q, m, req);
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
      if (v >= (uint32_t)n) {
        bad = true;
      } else {
        const uint32_t bit = 1u << (v & 31u);
        const uint32_t old = atomicOr(&bitmap[v >> 5], bit);
        if (old & bit) bad = true;
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
    int64_t *drow = DETAIL ? detail + row * n * 2 : nullptr;
    const Score s = ls ? ((m.flags & kFlagNarrowTime) ? replay_cont_ls<DETAIL, true>(m, req, perm, Remap{0, 0, 0}, scratch, drow)
                                                      : replay_cont_ls<DETAIL, false>(m, req, perm, Remap{0, 0, 0}, scratch, drow))
                       : replay_any<DETAIL>(m, req, perm, Remap{0, 0, 0}, stage, drow);
    if (lane == 0) {
      out[2 * row] = s.n;
      out[2 * row + 1] = (int64_t)s.t;
    }
    wave_sync_lds();
  }
}

__device__ __forceinline__ bool key_better(int64_t n1, uint64_t t1, int64_t n2, uint64_t t2) {
  return n1 > n2 || (n1 == n2 && t1 < t2);
}

// Algorithm 1 initialisation by one workgroup of 1024 threads; n <= 1024.
__device__ void start_body(const DevModel &m, const QueuePtrs &q, int chains, int iters, int64_t t_ref_user,
                           const SearchParams &srch, unsigned char *ws) {
  __shared__ uint4 req[1024];
  __shared__ uint64_t key_solo[1024];
  __shared__ uint16_t key_id[1024];
  __shared__ uint16_t ident[1024];
  __shared__ uint4 stage[64];
  const int n = m.n;
  const int tid = threadIdx.x;
  load_requests(q, m, req);
  int np = 1;
  while (np < n) np <<= 1;
  if (tid < np) {
    if (tid < n) {
      const uint32_t lin = q.in_len[tid], L = q.out_len[tid];
      // a request replayed alone: prefill, then L decode steps at batch size 1 with
      // context l_in + k, k = 1..L
      key_solo[tid] = m.p0 + m.p1 * lin + (uint64_t)L * (m.d0 + m.d1 + m.d2 * lin) + m.d2 * ((uint64_t)L * (L + 1) / 2);
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
    const Score sorted = replay<false>(m, req, key_id, Remap{0, 0, 0}, stage, nullptr);
    const Score input = replay<false>(m, req, ident, Remap{0, 0, 0}, stage, nullptr);
    // the better of the two starts; with the early exit, a sorted order that meets every
    // SLO is the result itself
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
      h->policy = m.policy;
      h->max_batch = m.B;
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

// The first kernel of a single-queue annealing call: the device checks of the queue (their
// verdict goes to the header; a failed check ends the call here), then the start order.
__global__ void __launch_bounds__(1024) start_kernel(DevModel m, QueuePtrs q, int chains, int iters,
                                                      int64_t t_ref_user, SearchParams srch, unsigned char *ws) {
  const Plan p = plan_in_block(q, m);
  if (p.status != 0) {
    if (threadIdx.x == 0) write_failed_header(ws, p, m.n, chains, iters, m.policy, m.B);
    return;
  }
  if (threadIdx.x == 0) write_plan(ws, p);
  m.flags |= (int32_t)(p.flags & m.gate.allow);
  start_body(m, q, chains, iters, t_ref_user, srch, ws);
}

// One chain by one wave, full replay per proposal: the chain's record slot is `chain`, its
// random stream is Philox chain index `rng_chain`. wbase: the wave's LDS (current and
// candidate-scratch orders, replay staging); req: the request records in LDS.
template <int OBJ>
__device__ void anneal_chain_body(const DevModel &m, const uint4 *req, unsigned char *wbase, int chains, int chain,
                                  uint32_t rng_chain, int iters, double T0, double alpha, uint32_t key0, uint32_t key1,
                                  uint64_t swap_thr, const SearchParams &srch, unsigned char *ws) {
  const int n = m.n;
  uint16_t *bufA = reinterpret_cast<uint16_t *>(wbase);
  uint16_t *bufB = reinterpret_cast<uint16_t *>(wbase + lds_align((size_t)n * 2));
  uint4 *stage = reinterpret_cast<uint4 *>(wbase + 2 * lds_align((size_t)n * 2));
  const int lane = lane_id();
  const WsHeader *h = reinterpret_cast<const WsHeader *>(ws);
  const int64_t t_ref = h->t_ref;
  int64_t cn = h->start_n;
  uint64_t ct = (uint64_t)h->start_t;
  const int64_t allmet = h->allmet;
  const uint16_t *start = reinterpret_cast<const uint16_t *>(ws + ws_off_start());
  const size_t stride = ws_perm_stride(n);
  uint16_t *gbest = reinterpret_cast<uint16_t *>(ws + ws_off_best(n, chains)) + (size_t)chain * stride;
  uint16_t *gcur = reinterpret_cast<uint16_t *>(ws + ws_off_cur(n, chains)) + (size_t)chain * stride;
  for (int p = lane; p < n; p += kWave) {
    const uint16_t v = start[p];
    bufA[p] = v;
    gbest[p] = v;
  }
  wave_sync_lds();
  uint16_t *cur = bufA, *cand = bufB;
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
    const Remap rm{(int)((pk >> 20) & 1u) + 1, i, j};
    const Score s = replay_any<false>(m, req, cur, rm, stage, nullptr);
    const bool acc = obj_accept<OBJ>(cn, ct, s.n - cn, (int64_t)(s.t - ct), t_ref, cool.T, w3);
    if (acc) {
      for (int p = lane; p < n; p += kWave) cand[p] = cur[rm.src(p)];
      wave_sync_lds();
      uint16_t *tmp = cur;
      cur = cand;
      cand = tmp;
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
        for (int p = lane; p < n; p += kWave) gbest[p] = cur[p];
      }
    }
    cool.step();
  }
  for (int p = lane; p < n; p += kWave) gcur[p] = cur[p];
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

// Per-wave LDS: current and candidate-scratch orders, replay staging.
template <int OBJ>
__global__ void __launch_bounds__(kBlock) anneal_kernel(DevModel m, QueuePtrs q, int chains, int iters, double T0,
                                                         double alpha, uint32_t key0, uint32_t key1,
                                                         uint64_t swap_thr, SearchParams srch, unsigned char *ws) {
  extern __shared__ __align__(16) unsigned char lds[];
  if (!gate_open(ws, m.gate, m.flags)) return;
  const int n = m.n;
  uint4 *req = reinterpret_cast<uint4 *>(lds);
  const size_t per_wave = lds_align((size_t)n * 2) * 2 + 64 * 16;
  const int wave = uniform((int)(threadIdx.x >> 6));
  unsigned char *wbase = lds + lds_align((size_t)n * 16) + (size_t)wave * per_wave;
  load_requests(q, m, req);
  __syncthreads();
  const int chain = uniform((int)blockIdx.x * kWavesPerBlock + wave);
  if (chain >= chains) return;
  anneal_chain_body<OBJ>(m, req, wbase, chains, chain, (uint32_t)chain, iters, T0, alpha, key0, key1, swap_thr, srch,
                         ws);
}

// Continuous admission: one wave per chain, blockDim / 64 chains per workgroup. Every
// proposal is replayed from the start, by list scheduling and scans (LS) or by the event
// loop; the candidate order is read through a remap of the current one and an accepted
// move is applied in place.
template <bool LS, int OBJ>
__global__ void __launch_bounds__(1024) anneal_cont_kernel(DevModel m, QueuePtrs q, int chains, int iters, double T0,
                                                            double alpha, uint32_t key0, uint32_t key1,
                                                            uint64_t swap_thr, SearchParams srch, unsigned char *ws) {
  extern __shared__ __align__(16) unsigned char lds[];
  if (!gate_open(ws, m.gate, m.flags)) return;
  const int n = m.n;
  const int waves = blockDim.x >> 6;
  uint4 *req = reinterpret_cast<uint4 *>(lds);
  const int wave = uniform((int)(threadIdx.x >> 6));
  // with at most 32 running requests the list-scheduling replay restarts at the first
  // changed admission, keeping the current order's pops and chunk-start keys
  const bool inc = LS && min(m.B, n) <= 32;
  const size_t ls_b = LS ? lds_align(cont_ls_scratch_bytes(n)) : 0;
  const size_t per_wave = lds_align((size_t)n * 2) + ls_b + (inc ? cont_inc_bytes(n, m.B) : 0);
  uint16_t *perm = reinterpret_cast<uint16_t *>(lds + lds_align((size_t)n * 16) + (size_t)wave * per_wave);
  unsigned char *scratch = reinterpret_cast<unsigned char *>(perm) + lds_align((size_t)n * 2);
  load_requests(q, m, req);
  __syncthreads();
  const int chain = uniform((int)blockIdx.x * waves + wave);
  if (chain >= chains) return;
  const int lane = lane_id();
  const WsHeader *h = reinterpret_cast<const WsHeader *>(ws);
  const int64_t t_ref = h->t_ref;
  int64_t cn = h->start_n;
  uint64_t ct = (uint64_t)h->start_t;
  const int64_t allmet = h->allmet;
  const uint16_t *start = reinterpret_cast<const uint16_t *>(ws + ws_off_start());
  const size_t stride = ws_perm_stride(n);
  uint16_t *gbest = reinterpret_cast<uint16_t *>(ws + ws_off_best(n, chains)) + (size_t)chain * stride;
  uint16_t *gcur = reinterpret_cast<uint16_t *>(ws + ws_off_cur(n, chains)) + (size_t)chain * stride;
  for (int p = lane; p < n; p += kWave) {
    const uint16_t v = start[p];
    perm[p] = v;
    gbest[p] = v;
  }
  wave_sync_lds();
  const bool narrow_t = (m.flags & kFlagNarrowTime) != 0;
  LsCache cache{};
  if (inc) {
    unsigned char *ib = scratch + ls_b;
    const size_t evb = ((size_t)4 * n + 15) / 16 * 16, snapb = (cont_inc_bytes(n, m.B) - 2 * evb) / 2;
    cache.ev_cur = reinterpret_cast<uint32_t *>(ib);
    cache.ev_cand = reinterpret_cast<uint32_t *>(ib + evb);
    cache.snap_cur = reinterpret_cast<uint32_t *>(ib + 2 * evb);
    cache.snap_cand = reinterpret_cast<uint32_t *>(ib + 2 * evb + snapb);
    // the start order's records by position and its state
    uint4 *posr = reinterpret_cast<uint4 *>(scratch + cont_ls_off_pos(n));
    for (int p = lane; p < n; p += kWave) posr[p] = req[perm[p]];
    wave_sync_lds();
    cache.lo = 0;
    if (narrow_t)
      replay_cont_ls<false, true, true>(m, req, perm, Remap{0, 0, 0}, scratch, nullptr, &cache);
    else
      replay_cont_ls<false, false, true>(m, req, perm, Remap{0, 0, 0}, scratch, nullptr, &cache);
    cache.accept();
  }
  int64_t bn = cn;
  uint64_t bt = ct;
  int64_t biter = -1, accepts = 0;
  uint64_t digest = kFnvOffset;
  Cooling cool{T0, alpha, srch.level_len, srch.level_len};
  ProposalStream ps;
  const int iters_run = (srch.early_exit && allmet) ? 0 : iters;
  for (int k = 0; k < iters_run; ++k) {
    if ((k & (kWave - 1)) == 0) ps.refill(k, lane, n, (uint32_t)chain, key0, key1, swap_thr, 0);
    const uint32_t pk = ps.packed(k), w3 = ps.word3(k);
    const int i = (int)(pk & 1023u), j = (int)((pk >> 10) & 1023u);
    const Remap rm{(int)((pk >> 20) & 1u) + 1, i, j};
    Score s;
    if (inc) {
      apply_move_lds(reinterpret_cast<uint4 *>(scratch + cont_ls_off_pos(n)), i == j ? 0 : rm.kind, i, j, lane);
      cache.lo = min(i, j);
      s = narrow_t ? replay_cont_ls<false, true, true>(m, req, perm, rm, scratch, nullptr, &cache)
                   : replay_cont_ls<false, false, true>(m, req, perm, rm, scratch, nullptr, &cache);
    } else {
      s = LS ? (narrow_t ? replay_cont_ls<false, true>(m, req, perm, rm, scratch, nullptr)
                         : replay_cont_ls<false, false>(m, req, perm, rm, scratch, nullptr))
             : replay_cont_fast<false>(m, req, perm, rm, nullptr);
    }
    const bool acc = obj_accept<OBJ>(cn, ct, s.n - cn, (int64_t)(s.t - ct), t_ref, cool.T, w3);
    if (inc && !acc) apply_move_lds(reinterpret_cast<uint4 *>(scratch + cont_ls_off_pos(n)), i == j ? 0 : rm.kind, j, i, lane);
    if (acc) {
      apply_move_lds(perm, i == j ? 0 : rm.kind, i, j, lane);
      if (inc) cache.accept();
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
        for (int p = lane; p < n; p += kWave) gbest[p] = perm[p];
      }
    }
    cool.step();
  }
  for (int p = lane; p < n; p += kWave) gcur[p] = perm[p];
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

// One workgroup of 1024 threads: argmax over chains of the best key (lowest chain id
// among equals).
__device__ void reduce_body(unsigned char *ws) {
  __shared__ int64_t sn[1024];
  __shared__ uint64_t st[1024];
  __shared__ int32_t sc[1024];
  WsHeader *h = reinterpret_cast<WsHeader *>(ws);
  const int n = h->n, chains = h->chains;
  const int64_t *rec = reinterpret_cast<const int64_t *>(ws + ws_off_records(n));
  const bool ratio = h->objective != 0;
  // a chain wins over another iff its best key is strictly better, or neither is better
  // and its id is lower
  auto wins = [ratio](int64_t n1, uint64_t t1, int32_t c1, int64_t n2, uint64_t t2, int32_t c2) {
    if (c2 == 0x7FFFFFFF) return c1 != 0x7FFFFFFF;
    if (c1 == 0x7FFFFFFF) return false;
    const bool b12 = ratio ? obj_better<1>(n1, t1, n2, t2) : obj_better<0>(n1, t1, n2, t2);
    const bool b21 = ratio ? obj_better<1>(n2, t2, n1, t1) : obj_better<0>(n2, t2, n1, t1);
    return b12 || (!b21 && c1 < c2);
  };
  int64_t bn = -1;
  uint64_t bt = ~0ull;
  int32_t bc = 0x7FFFFFFF;
  for (int c = threadIdx.x; c < chains; c += blockDim.x) {
    const int64_t cn = rec[(size_t)c * 8 + 2];
    const uint64_t ctt = (uint64_t)rec[(size_t)c * 8 + 3];
    if (wins(cn, ctt, c, bn, bt, bc)) {
      bn = cn;
      bt = ctt;
      bc = c;
    }
  }
  sn[threadIdx.x] = bn;
  st[threadIdx.x] = bt;
  sc[threadIdx.x] = bc;
  __syncthreads();
  for (int o = blockDim.x / 2; o > 0; o >>= 1) {
    if ((int)threadIdx.x < o) {
      const int u = threadIdx.x + o;
      if (wins(sn[u], st[u], sc[u], sn[threadIdx.x], st[threadIdx.x], sc[threadIdx.x])) {
        sn[threadIdx.x] = sn[u];
        st[threadIdx.x] = st[u];
        sc[threadIdx.x] = sc[u];
      }
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) {
    h->best_chain = sc[0];
    h->best_n = sn[0];
    h->best_t = (int64_t)st[0];
  }
}

__global__ void __launch_bounds__(1024) reduce_kernel(unsigned char *ws) {
  if (!plan_ok(ws)) return;
  reduce_body(ws);
}

// After a call whose queue failed the device checks the key reads (-2, code, -1) and the
// order is left as it is.
__global__ void __launch_bounds__(256) best_copy_kernel(const unsigned char *ws, uint16_t *perm_out, int64_t *key_out) {
  const WsHeader *h = reinterpret_cast<const WsHeader *>(ws);
  if (h->plan_status != 0) {
    if (threadIdx.x == 0) {
      key_out[0] = -2;
      key_out[1] = h->plan_status;
      key_out[2] = -1;
    }
    return;
  }
  const int n = h->n, chains = h->chains;
  const int64_t c = h->best_chain;
  const uint16_t *src = reinterpret_cast<const uint16_t *>(ws + ws_off_best(n, chains)) + (size_t)c * ws_perm_stride(n);
  for (int p = threadIdx.x; p < n; p += blockDim.x) perm_out[p] = src[p];
  if (threadIdx.x == 0) {
    key_out[0] = h->best_n;
    key_out[1] = h->best_t;
    key_out[2] = c;
  }
}

// After a call whose queue failed the device checks every record reads (-2, code, -1, ...)
// and the orders are left as they are.
__global__ void __launch_bounds__(256) chains_copy_kernel(const unsigned char *ws, int64_t *per_chain, uint16_t *cur_out,
                                                           uint16_t *best_out) {
  const WsHeader *h = reinterpret_cast<const WsHeader *>(ws);
  const int n = h->n, chains = h->chains;
  if (h->plan_status != 0) {
    const int64_t status = h->plan_status;
    for (int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; u < (int64_t)chains * 8;
         u += (int64_t)gridDim.x * blockDim.x) {
      const int w = (int)(u & 7);
      per_chain[u] = w == 0 ? -2 : (w == 1 ? status : -1);
    }
    return;
  }
  const size_t stride = ws_perm_stride(n);
  const int64_t *rec = reinterpret_cast<const int64_t *>(ws + ws_off_records(n));
  const uint16_t *cur = reinterpret_cast<const uint16_t *>(ws + ws_off_cur(n, chains));
  const uint16_t *best = reinterpret_cast<const uint16_t *>(ws + ws_off_best(n, chains));
  const int64_t total = (int64_t)chains * 8;
  for (int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; u < total; u += (int64_t)gridDim.x * blockDim.x)
    per_chain[u] = rec[u];
  const int64_t tp = (int64_t)chains * n;
  for (int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; u < tp; u += (int64_t)gridDim.x * blockDim.x) {
    const int64_t c = u / n, p = u - c * n;
    if (cur_out) cur_out[u] = cur[c * stride + p];
    if (best_out) best_out[u] = best[c * stride + p];
  }
}

// After a call whose queue failed the device checks info reads (-2, code, -1, -1) and the
// order is left as it is.
__global__ void __launch_bounds__(256) start_copy_kernel(const unsigned char *ws, uint16_t *start_out, int64_t *info) {
  const WsHeader *h = reinterpret_cast<const WsHeader *>(ws);
  const int n = h->n;
  if (h->plan_status != 0) {
    if (threadIdx.x == 0) {
      info[0] = -2;
      info[1] = h->plan_status;
      info[2] = -1;
      info[3] = -1;
    }
    return;
  }
  const uint16_t *src = reinterpret_cast<const uint16_t *>(ws + ws_off_start());
  for (int p = threadIdx.x; p < n; p += blockDim.x) start_out[p] = src[p];
  if (threadIdx.x == 0) {
    info[0] = h->t_ref;
    info[1] = h->start_n;
    info[2] = h->start_t;
    info[3] = h->allmet;
  }
}

// The device checks' verdict of the last call on a workspace (single-queue or several
// instances: the fields sit at the same offsets): status, width flags, selected kernel.
__global__ void status_copy_kernel(const unsigned char *ws, int64_t *out) {
  const WsHeader *h = reinterpret_cast<const WsHeader *>(ws);
  out[0] = h->plan_status;
  out[1] = h->plan_flags;
  out[2] = h->plan_selected;
}

// One thread per row: Durstenfeld's in-place Fisher-Yates, drawing from Philox.
__global__ void __launch_bounds__(256) shuffle_kernel(uint32_t key0, uint32_t key1, int n, int64_t row0, int64_t rows,
                                                       uint16_t *perms) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= rows) return;
  const uint32_t idx = (uint32_t)(row0 + t);
  uint16_t *p = perms + t * n;
  for (int u = 0; u < n; ++u) p[u] = (uint16_t)u;
  u32x4 w{0, 0, 0, 0};
  for (int k = n - 1; k >= 1; --k) {
    if (k == n - 1 || (k & 3) == 3) w = philox4x32_10((uint32_t)k >> 2, idx, 1u, kTagShuffle, key0, key1);
    const uint32_t word = (k & 3) == 0 ? w.x : (k & 3) == 1 ? w.y : (k & 3) == 2 ? w.z : w.w;
    const uint32_t j = (uint32_t)(((uint64_t)word * (uint64_t)(k + 1)) >> 32);
    const uint16_t a = p[k];
    p[k] = p[j];
    p[j] = a;
  }
}

// The acceptance rule of the annealing kernels on given inputs, one element per thread:
// rule 0 is metropolis(a, b, T, w3), rule 1 metropolis_ratio(a, b, c, d, T, w3); out holds
// the decision in bit 0 and whether the single-precision screen took it in bit 1.
__global__ void __launch_bounds__(256) accept_check_kernel(int rule, int64_t k, const int64_t *__restrict__ a,
                                                           const int64_t *__restrict__ b,
                                                           const uint64_t *__restrict__ c,
                                                           const uint64_t *__restrict__ d,
                                                           const double *__restrict__ T,
                                                           const uint32_t *__restrict__ w3, uint8_t *__restrict__ out) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t r = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; r < k; r += stride) {
    const int v = rule == 1 ? metropolis_ratio_rule(a[r], b[r], c[r], d[r], T[r], w3[r])
                            : metropolis_rule(a[r], b[r], T[r], w3[r]);
    out[r] = (uint8_t)v;
  }
}

}  // namespace sa
