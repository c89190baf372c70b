// Joint search over the priority order and the static batch sizes (gfx950, wave64).
//
// The Problem Formulation makes the batch sizes b_0 .. b_{M-1} (sum N, each at most the
// maximum) part of the decision next to the order, and Algorithm 1 explores them with two
// moves besides the swap: squeezeLastIter puts a request into the batch that runs just
// before its own (when that one is below the maximum size), delayNextIter into the batch
// that runs just after (when that one is below the maximum, or a new last batch when the
// request does not run alone). The three moves are drawn uniformly: move = floor(w0 * 3 /
// 2^32), 0 squeeze and 1 delay at position i, 2 swap of positions i and j.
//
// The layout is one start flag per position (1 where a batch begins, position 0 always).
// A moved request takes the adjoining end of its new batch: the previous batch's last
// position (an insert from i to the first position of its batch) or the next batch's
// first position (an insert from i to the last position of its batch); the flags of the
// two batch ends move with it. A move that is not allowed changes nothing and is neither
// accepted nor rejected. Every chain starts from the start order with maximum-size
// batches.
//
// This file holds the layout helpers, the full replay with explicit batches (64-bit, any
// widths), the evaluation kernel over K (order, layout) rows and the full-replay annealing
// kernel. The delta kernel for queues whose timelines fit 32 bits is further below.
#pragma once
#include "device_common.h"
#include "device_replay.h"
#include "device_rng.h"
#include "anneal_static.h"
#include "kernels.h"

namespace sa {

// First position after p that begins a batch, or n. Valid layouts have batches of at most
// 64 positions, so one of the 64 positions read holds it (the clamps only keep a malformed
// layout inside the arrays).
__device__ __forceinline__ int batch_end(const uint8_t *f, int n, int p, int lane) {
  const int q = p + 1 + lane;
  const bool st = q >= n || f[min(q, n - 1)] != 0;
  const uint64_t b = __ballot(st);
  return min(n, p + 1 + (b ? (int)__builtin_ctzll(b) : 63));
}
// Position that begins the batch holding p.
__device__ __forceinline__ int batch_begin(const uint8_t *f, int p, int lane) {
  const int q = p - lane;
  const bool st = q <= 0 || f[max(q, 0)] != 0;
  return p - (int)__builtin_ctzll(__ballot(st));
}

// Valid layout: flags in {0, 1}, position 0 begins a batch, every batch holds at most B
// positions (no position lies B or more past the last start at or before it).
__device__ bool layout_ok(const uint8_t *f, int n, int B, int lane) {
  bool bad = false;
  int carry = 0;
  for (int c0 = 0; c0 < n; c0 += kWave) {
    const int p = c0 + lane;
    const uint32_t v = p < n ? f[p] : 1u;
    bad |= v > 1u || (p == 0 && v != 1u);
    int last = (p < n && v == 1u) ? p : -1;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
      const int y = __shfl_up(last, o);
      if (lane >= o) last = max(last, y);
    }
    last = max(last, carry);
    bad |= p < n && p - last >= B;
    carry = __shfl(last, kWave - 1);
  }
  return __ballot(bad) == 0ull;
}

__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = max(v, (uint64_t)__shfl_xor(v, o));
  return v;
}

// Static timeline with explicit batches, one batch at a time: the members occupy lanes
// 0 .. b-1; member m's finish offset within its batch is the batch prefill plus its own
// L_m decode iterations, each costing d0 + d1 * (members still decoding) + d2 * (their
// contexts), summed in closed form over every member j it shares mu = min(L_j, L_m)
// iterations with:
//   F_m = P + L_m d0 + sum_j [ d1 mu + d2 (l_j mu + mu (mu + 1) / 2) ].
// The batch lasts max F; the next batch starts when it ends (waiting time = sum of the
// earlier batch durations).
template <bool DETAIL>
__device__ Score replay_batches(const DevModel &m, const uint4 *__restrict__ req, const uint16_t *perm,
                                const uint8_t *flags, uint4 *stage, int64_t *detail) {
  const int lane = lane_id();
  const int n = m.n;
  uint64_t S = 0, tl = 0;
  int64_t nmet = 0;
  for (int s = 0; s < n;) {
    const int e = batch_end(flags, n, s, lane);
    const int b = e - s;
    const bool valid = lane < b;
    uint32_t lin = 0, L = 0, thr = 0, kind = 0;
    int r = 0;
    if (valid) {
      r = perm[s + lane];
      const uint4 rq = req[r];
      lin = req_lin(rq);
      L = req_lout(rq);
      thr = rq.y;
      kind = rq.z & 3u;
    }
    const uint64_t pf = valid ? m.p0 + m.p1 * (uint64_t)lin : 0;
    stage[lane] = make_uint4(L, lin, (uint32_t)pf, (uint32_t)(pf >> 32));
    wave_sync_lds();
    uint64_t P = 0, acc = 0;
    for (int j = 0; j < b; ++j) {
      const uint4 sj = stage[j];
      P += (uint64_t)sj.z | ((uint64_t)sj.w << 32);
      const uint64_t mu = min(sj.x, L);
      acc += m.d1 * mu + m.d2 * ((uint64_t)sj.y * mu + (mu * (mu + 1) >> 1));
    }
    wave_sync_lds();
    const uint64_t F = P + (uint64_t)L * m.d0 + acc;
    const uint64_t D = wave_max_u64(valid ? F : 0);
    bool met = false;
    if (valid) {
      const uint64_t e2e = S + F, ttft = S + P;
      tl += e2e;
      met = slo_met(kind, thr, L, ttft, e2e);
      if (DETAIL) {
        detail[2 * r] = (int64_t)ttft;
        detail[2 * r + 1] = (int64_t)e2e;
      }
    }
    nmet += ballot_count(met);
    S += D;
    s = e;
  }
  return Score{nmet, wave_sum_u64(tl)};
}

// K rows of (order, layout): one wave per row, rows validated first ((-1, -1) otherwise).
template <bool DETAIL>
__global__ void __launch_bounds__(256) eval_sized_kernel(DevModel m, QueuePtrs q, const uint16_t *__restrict__ perms,
                                                          const uint8_t *__restrict__ starts, int64_t rows,
                                                          int64_t *__restrict__ out, int64_t *__restrict__ detail) {
  extern __shared__ __align__(16) unsigned char lds[];
  const int n = m.n;
  uint4 *req = reinterpret_cast<uint4 *>(lds);
  const size_t pb = ((size_t)n * 2 + 15) & ~size_t(15), fb = ((size_t)n + 15) & ~size_t(15);
  const size_t per_wave = pb + fb + 64 * 16 + 32 * 4;
  const int wave = uniform((int)(threadIdx.x >> 6));
  unsigned char *wb = lds + (((size_t)n * 16 + 15) & ~size_t(15)) + (size_t)wave * per_wave;
  uint16_t *perm = reinterpret_cast<uint16_t *>(wb);
  uint8_t *flags = wb + pb;
  uint4 *stage = reinterpret_cast<uint4 *>(wb + pb + fb);
  uint32_t *bitmap = reinterpret_cast<uint32_t *>(wb + pb + fb + 64 * 16);
  for (int r = threadIdx.x; r < n; r += blockDim.x) {
    const uint32_t lin = q.in_len[r], lout = q.out_len[r];
    req[r] = make_uint4(lin | (lout << 16), q.thr[r], (uint32_t)q.kind[r], 0u);
  }
  __syncthreads();
  const int lane = lane_id();
  const int waves = blockDim.x >> 6;
  for (int64_t row = (int64_t)blockIdx.x * waves + wave; row < rows; row += (int64_t)gridDim.x * waves) {
    const uint16_t *src = perms + row * n;
    const uint8_t *fsrc = starts + row * n;
    if (lane < 32) bitmap[lane] = 0u;
    wave_sync_lds();
    bool bad = false;
    for (int p = lane; p < n; p += kWave) {
      const uint32_t v = src[p];
      perm[p] = (uint16_t)v;
      flags[p] = fsrc[p];
      if (v >= (uint32_t)n) {
        bad = true;
      } else {
        const uint32_t bit = 1u << (v & 31u);
        const uint32_t old = atomicOr(&bitmap[v >> 5], bit);
        if (old & bit) bad = true;
      }
    }
    wave_sync_lds();
    const bool ok = __ballot(bad) == 0ull && layout_ok(flags, n, m.B, lane);
    if (!ok) {
      if (lane == 0) {
        out[2 * row] = -1;
        out[2 * row + 1] = -1;
      }
      continue;
    }
    const Score s = replay_batches<DETAIL>(m, req, perm, flags, stage, DETAIL ? detail + row * n * 2 : nullptr);
    if (lane == 0) {
      out[2 * row] = s.n;
      out[2 * row + 1] = (int64_t)s.t;
    }
    wave_sync_lds();
  }
}

// Proposal draws of the joint search, 64 iterations per Philox pass (lane l: iteration
// k0 + l, counter (k0 + l, chain, 0, kTagAnneal)): i | j << 10 | move << 20, with i, j the
// swap positions (i alone for squeeze and delay) and move = floor(w0 * 3 / 2^32).
struct SizedDraws {
  uint32_t pk = 0, w3 = 0;
  __device__ __forceinline__ void refill(int k0, int lane, int n, uint32_t chain, uint32_t key0, uint32_t key1) {
    const u32x4 w = philox4x32_10((uint32_t)(k0 + lane), chain, 0u, kTagAnneal, key0, key1);
    int i, j;
    pick_positions(n, w.y, w.z, i, j);
    const uint32_t op = (uint32_t)(((uint64_t)w.x * 3u) >> 32);
    pk = (uint32_t)i | ((uint32_t)j << 10) | (op << 20);
    w3 = w.w;
  }
  __device__ __forceinline__ uint32_t packed(int k) const { return (uint32_t)__builtin_amdgcn_readlane((int)pk, k & 63); }
  __device__ __forceinline__ uint32_t word3(int k) const { return (uint32_t)__builtin_amdgcn_readlane((int)w3, k & 63); }
};

// Where a move takes the layout, from the current flags (all wave-uniform). The candidate
// order is the current one with an insert from i to `to` (squeeze, delay) or a swap of i
// and j; the flags change at the two batch ends. made == false: not allowed.
struct SizedMove {
  bool made;
  int op, i, j, to;
  int set0, clr0;  // flag writes: position set0 becomes a start (-1: none), clr0 stops being one (-1: none)
};

__device__ __forceinline__ SizedMove plan_move(const uint8_t *f, int n, int B, int op, int i, int j, int lane) {
  SizedMove mv{false, op, i, j, i, -1, -1};
  if (op == 2) {
    mv.made = n >= 2;
    return mv;
  }
  const int s = batch_begin(f, i, lane), e = batch_end(f, n, i, lane);
  if (op == 0) {
    if (s == 0) return mv;
    const int sp = batch_begin(f, s - 1, lane);
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
  const int en = batch_end(f, n, e, lane);
  if (en - e >= B) return mv;
  mv.made = true;
  mv.to = e - 1;
  mv.set0 = e - 1;
  mv.clr0 = e;
  return mv;
}

// Applies a planned move to an order and its flags in LDS (one wave).
__device__ __forceinline__ void apply_sized_move(uint16_t *perm, uint8_t *f, const SizedMove &mv, int lane) {
  if (mv.op == 2) {
    apply_move_lds(perm, 1, mv.i, mv.j, lane);
    return;
  }
  apply_move_lds(perm, 2, mv.i, mv.to, lane);
  if (lane == 0) {
    if (mv.clr0 >= 0) f[mv.clr0] = 0;
    if (mv.set0 >= 0) f[mv.set0] = 1;
  }
  wave_sync_lds();
}

__device__ __forceinline__ void write_record(unsigned char *ws, int n, int chain, int64_t cn, uint64_t ct, int64_t bn,
                                             uint64_t bt, int64_t biter, int64_t accepts, uint64_t digest,
                                             int64_t allmet) {
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

// Full replay per proposal (any widths): one wave per chain; per wave LDS holds the
// current and candidate orders and flags and the replay staging.
__global__ void __launch_bounds__(256) anneal_sized_generic_kernel(DevModel m, QueuePtrs q, int chains, int iters,
                                                                    double T0, double alpha, uint32_t key0,
                                                                    uint32_t key1, unsigned char *ws) {
  extern __shared__ __align__(16) unsigned char lds[];
  const int n = m.n, B = m.B;
  uint4 *req = reinterpret_cast<uint4 *>(lds);
  const size_t pb = ((size_t)n * 2 + 15) & ~size_t(15), fb = ((size_t)n + 15) & ~size_t(15);
  const size_t per_wave = 2 * pb + 2 * fb + 64 * 16;
  const int wave = uniform((int)(threadIdx.x >> 6));
  const int waves = blockDim.x >> 6;
  unsigned char *wb = lds + (((size_t)n * 16 + 15) & ~size_t(15)) + (size_t)wave * per_wave;
  uint16_t *cur = reinterpret_cast<uint16_t *>(wb);
  uint16_t *cand = reinterpret_cast<uint16_t *>(wb + pb);
  uint8_t *fcur = wb + 2 * pb, *fcand = wb + 2 * pb + fb;
  uint4 *stage = reinterpret_cast<uint4 *>(wb + 2 * pb + 2 * fb);
  for (int r = threadIdx.x; r < n; r += blockDim.x) {
    const uint32_t lin = q.in_len[r], lout = q.out_len[r];
    req[r] = make_uint4(lin | (lout << 16), q.thr[r], (uint32_t)q.kind[r], 0u);
  }
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
  double T = T0;
  SizedDraws ds;
  for (int k = 0; k < iters; ++k) {
    if ((k & (kWave - 1)) == 0) ds.refill(k, lane, n, (uint32_t)chain, key0, key1);
    const uint32_t pk = ds.packed(k), w3 = ds.word3(k);
    const SizedMove mv = plan_move(fcur, n, B, (int)(pk >> 20), (int)(pk & 1023u), (int)((pk >> 10) & 1023u), lane);
    if (mv.made) {
      for (int p = lane; p < n; p += kWave) {
        cand[p] = cur[p];
        fcand[p] = fcur[p];
      }
      wave_sync_lds();
      apply_sized_move(cand, fcand, mv, lane);
      const Score s = replay_batches<false>(m, req, cand, fcand, stage, nullptr);
      const int64_t delta = (s.n - cn) * t_ref - (int64_t)(s.t - ct);
      if (metropolis(delta, t_ref, T, w3)) {
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
        if (key_better(cn, ct, bn, bt)) {
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
    T = T * alpha;
  }
  for (int p = lane; p < n; p += kWave) {
    gcur[p] = cur[p];
    gcur_f[p] = fcur[p];
  }
  if (lane == 0) write_record(ws, n, chain, cn, ct, bn, bt, biter, accepts, digest, allmet);
}

// Readouts of the layouts: per chain current and best flags, and the best chain's.
__global__ void __launch_bounds__(256) starts_copy_kernel(const unsigned char *ws, uint8_t *cur_out, uint8_t *best_out,
                                                           uint8_t *winner_out) {
  const WsHeader *h = reinterpret_cast<const WsHeader *>(ws);
  const int n = h->n, chains = h->chains, B = (int)h->max_batch;
  const bool searched = h->policy == 2;  // other policies keep maximum-size batches
  const size_t fs = ws_flag_stride(n);
  const uint8_t *cur = ws + ws_off_cur_starts(n, chains);
  const uint8_t *best = ws + ws_off_best_starts(n, chains);
  const int64_t tp = (int64_t)chains * n;
  for (int64_t u = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; u < tp; u += (int64_t)gridDim.x * blockDim.x) {
    const int64_t c = u / n, p = u - c * n;
    if (cur_out) cur_out[u] = searched ? cur[c * fs + p] : (uint8_t)(p % B == 0);
    if (best_out) best_out[u] = searched ? best[c * fs + p] : (uint8_t)(p % B == 0);
  }
  if (winner_out && blockIdx.x == 0) {
    const int64_t c = h->best_chain;
    for (int p = threadIdx.x; p < n; p += blockDim.x) winner_out[p] = searched ? best[c * fs + p] : (uint8_t)(p % B == 0);
  }
}

}  // namespace sa
