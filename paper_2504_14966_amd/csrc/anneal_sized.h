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
#include <utility>
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
__device__ Score replay_batches_one(const DevModel &m, const uint4 *__restrict__ req, const uint16_t *perm,
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

// The same timeline over windows of whole batches, one position per lane: a window starts
// at a batch start and takes every batch that ends within the next 64 positions. Each lane
// sums its pair terms over its own batch's members from the staged records (as many steps
// as the window's largest batch), which also gives the batch prefill. Batch durations are
// one max-scan of (first lane of the batch << 58 | finish offset) -- first lanes never
// decrease across lanes, so the running maximum at a lane is the running maximum within its
// own batch -- and the start times one add-scan of the durations at the batch-last lanes.
// Needs every time below 2^58 (kFlagWindows).
template <bool DETAIL>
__device__ Score replay_batches_windows(const DevModel &m, const uint4 *__restrict__ req, const uint16_t *perm,
                                        const uint8_t *flags, uint4 *stage, int64_t *detail) {
  const int lane = lane_id();
  const int n = m.n;
  constexpr uint64_t kTimeMask = (uint64_t(1) << 58) - 1;
  uint64_t S0 = 0, tl = 0;
  int64_t nmet = 0;
  for (int s = 0; s < n;) {
    const int p = s + lane;
    const bool st = p == n || (p < n && (lane == 0 || flags[p] != 0));  // begins a batch, or the end
    bool st64 = s + kWave == n;                                         // position s + 64 likewise
    if (s + kWave < n) st64 = flags[s + kWave] != 0;
    uint64_t lastm = (__ballot(st) >> 1) | (st64 ? uint64_t(1) << 63 : 0ull);  // batch-last lanes
    // a valid layout always closes a batch within 64 positions; a malformed one is cut
    // there so that the window advances
    if (lastm == 0ull) lastm = uint64_t(1) << 63;
    const int w = 64 - __clzll(lastm);
    const bool in = lane < w;
    const uint64_t below = lastm & ((uint64_t(1) << lane) - 1);
    const int b0 = below ? 64 - __clzll(below) : 0;
    const int b1 = lane + __builtin_ctzll(in ? (lastm >> lane) : 1ull);
    uint32_t lin = 0, L = 0, thr = 0, kind = 0;
    int r = 0;
    if (in) {
      r = perm[p];
      const uint4 rq = req[r];
      lin = req_lin(rq);
      L = req_lout(rq);
      thr = rq.y;
      kind = rq.z & 3u;
    }
    const uint64_t pf = in ? m.p0 + m.p1 * (uint64_t)lin : 0;
    const bool narrow = (m.flags & kFlagStaticNarrow) != 0;
    // narrow widths stage the pair-cost parameter e = 2 (d1 + d2 l_in) + d2 instead of l_in
    const uint32_t ev = narrow ? (uint32_t)(2 * (m.d1 + m.d2 * lin) + m.d2) : lin;
    stage[lane] = make_uint4(L, ev, (uint32_t)pf, (uint32_t)(pf >> 32));
    wave_sync_lds();
    const int bl = in ? b1 - b0 + 1 : 0;
    int jmax = bl;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) jmax = max(jmax, __shfl_xor(jmax, o));
    uint64_t P = 0, acc = 0;
    if (narrow) {
      // doubled pair costs mu (e_j + d2 mu) in 24-bit products (each below 2^32, and their
      // sum over a batch too: the host's width check), halved once
      const uint32_t d2 = (uint32_t)m.d2;
      uint32_t acc2 = 0, P32 = 0;
      for (int j = 0; j < jmax; ++j) {
        if (j < bl) {
          const uint4 sj = stage[b0 + j];
          P32 += sj.z;
          const uint32_t mu = min(sj.x, L);
          acc2 = mad24_v(mu, mad24_v(d2, mu, sj.y), acc2);
        }
      }
      P = P32;
      acc = acc2 >> 1;
    } else {
      for (int j = 0; j < jmax; ++j) {
        if (j < bl) {
          const uint4 sj = stage[b0 + j];
          P += (uint64_t)sj.z | ((uint64_t)sj.w << 32);
          const uint64_t mu = min(sj.x, L);
          acc += m.d1 * mu + m.d2 * ((uint64_t)sj.y * mu + (mu * (mu + 1) >> 1));
        }
      }
    }
    wave_sync_lds();
    const uint64_t F = P + (uint64_t)L * m.d0 + acc;
    const uint64_t D = scan_max64(in ? ((uint64_t)b0 << 58) | F : 0ull) & kTimeMask;
    const uint64_t contrib = (in && lane == b1) ? D : 0ull;
    const uint64_t incl = scan_add64(contrib);
    const uint64_t S = S0 + (incl - contrib);
    bool met = false;
    if (in) {
      const uint64_t e2e = S + F, ttft = S + P;
      tl += e2e;
      met = slo_met(kind, thr, L, ttft, e2e);
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

// The same windows when the pair costs take the narrow widths and the whole timeline fits 32
// bits (kFlagStaticNarrow and kFlagTime32): 32-bit offsets, durations by the 32-bit max-scan
// confined to batches, starts by a 32-bit add-scan, the latency sum in 16-bit halves (each
// lane's below 2^26 over at most 1024 windows).
template <bool DETAIL>
__device__ Score replay_batches_windows32(const DevModel &m, const uint4 *__restrict__ req, const uint16_t *perm,
                                          const uint8_t *flags, uint4 *stage, int64_t *detail) {
  const int lane = lane_id();
  const int n = m.n;
  const uint32_t d0 = (uint32_t)m.d0, d2 = (uint32_t)m.d2;
  uint32_t S0 = 0, tlo = 0, thi = 0;
  int64_t nmet = 0;
  for (int s = 0; s < n;) {
    const int p = s + lane;
    const bool st = p == n || (p < n && (lane == 0 || flags[p] != 0));  // begins a batch, or the end
    bool st64 = s + kWave == n;                                         // position s + 64 likewise
    if (s + kWave < n) st64 = flags[s + kWave] != 0;
    uint64_t lastm = (__ballot(st) >> 1) | (st64 ? uint64_t(1) << 63 : 0ull);  // batch-last lanes
    if (lastm == 0ull) lastm = uint64_t(1) << 63;
    const int w = 64 - __clzll(lastm);
    const bool in = lane < w;
    const uint64_t below = lastm & ((uint64_t(1) << lane) - 1);
    const int b0 = below ? 64 - __clzll(below) : 0;
    const int b1 = lane + __builtin_ctzll(in ? (lastm >> lane) : 1ull);
    uint32_t lin = 0, L = 0, thr = 0, kind = 0;
    int r = 0;
    if (in) {
      r = perm[p];
      const uint4 rq = req[r];
      lin = req_lin(rq);
      L = req_lout(rq);
      thr = rq.y;
      kind = rq.z & 3u;
    }
    const uint32_t pf = in ? (uint32_t)(m.p0 + m.p1 * (uint64_t)lin) : 0u;
    stage[lane] = make_uint4(L, (uint32_t)(2 * (m.d1 + m.d2 * lin) + m.d2), pf, 0u);
    wave_sync_lds();
    const int bl = in ? b1 - b0 + 1 : 0;
    int jmax = bl;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) jmax = max(jmax, __shfl_xor(jmax, o));
    uint32_t acc2 = 0, P = 0;
    for (int j = 0; j < jmax; ++j) {
      if (j < bl) {
        const uint4 sj = stage[b0 + j];
        P += sj.z;
        const uint32_t mu = min(sj.x, L);
        acc2 = mad24_v(mu, mad24_v(d2, mu, sj.y), acc2);
      }
    }
    wave_sync_lds();
    const uint32_t F = in ? P + __umul24(L, d0) + (acc2 >> 1) : 0u;
    // lanes past the window hold F = 0 and send nothing; what they receive is unused
    const uint32_t D = seg_max32(F, b0, b1, lane);
    const uint32_t contrib = (in && lane == b1) ? D : 0u;
    const uint32_t incl = scan_add32(contrib);
    const uint32_t S = S0 + incl - contrib;
    bool met = false;
    if (in) {
      const uint32_t e2e = S + F, ttft = S + P;
      tlo += e2e & 0xFFFFu;
      thi += e2e >> 16;
      met = kind == 0 ? ttft <= thr : (kind == 2 ? e2e <= thr : (uint64_t)(F - P) <= (uint64_t)thr * L);
      if (DETAIL) {
        detail[2 * r] = (int64_t)ttft;
        detail[2 * r + 1] = (int64_t)e2e;
      }
    }
    nmet += ballot_count(met);
    S0 += readlane(incl, kWave - 1);
    s += w;
  }
  Seg<6>::template all2<OpAdd, OpAdd>(tlo, thi, lane);
  return Score{nmet, (uint64_t)tlo + ((uint64_t)thi << 16)};
}

template <bool DETAIL>
__device__ __forceinline__ Score replay_batches(const DevModel &m, const uint4 *__restrict__ req, const uint16_t *perm,
                                                const uint8_t *flags, uint4 *stage, int64_t *detail) {
  if ((m.flags & (kFlagStaticNarrow | kFlagTime32)) == (kFlagStaticNarrow | kFlagTime32))
    return replay_batches_windows32<DETAIL>(m, req, perm, flags, stage, detail);
  if (m.flags & kFlagWindows) return replay_batches_windows<DETAIL>(m, req, perm, flags, stage, detail);
  return replay_batches_one<DETAIL>(m, req, perm, flags, stage, detail);
}

// K rows of (order, layout): one wave per row, rows validated first ((-1, -1) otherwise).
template <bool DETAIL>
__global__ void __launch_bounds__(256) eval_sized_kernel(DevModel m, QueuePtrs q, const uint16_t *__restrict__ perms,
                                                          const uint8_t *__restrict__ starts, int64_t rows,
                                                          int64_t *__restrict__ out, int64_t *__restrict__ detail) {
  extern __shared__ __align__(16) unsigned char lds[];
  const EvalRows span = eval_gate(q, m, rows, out);
  if (span.end <= span.begin) return;
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
  for (int64_t row = span.begin + (int64_t)blockIdx.x * waves + wave; row < span.end;
       row += (int64_t)gridDim.x * waves) {
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
template <int OBJ>
__global__ void __launch_bounds__(256) anneal_sized_generic_kernel(DevModel m, QueuePtrs q, int chains, int iters,
                                                                    double T0, double alpha, uint32_t key0,
                                                                    uint32_t key1, SearchParams srch,
                                                                    unsigned char *ws) {
  extern __shared__ __align__(16) unsigned char lds[];
  if (!gate_open(ws, m.gate, m.flags)) return;
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
  Cooling cool{T0, alpha, srch.level_len, srch.level_len};
  SizedDraws ds;
  const int iters_run = (srch.early_exit && allmet) ? 0 : iters;
  for (int k = 0; k < iters_run; ++k) {
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

// ---- delta kernel: timelines that fit 32 bits ----
//
// Per chain (one wave). In LDS:
//   perm, flags   the current order and layout;
//   F[r]          request r's finish offset within its batch, prefill included (u32).
// In registers, position p in row p / 64, lane p % 64 (NR rows):
//   S             start time of the batch holding p (u32);
//   lim           the member at p meets its SLO iff S < lim (u32): thr - P + 1 for TTFT
//                 (P = batch prefill), thr - F + 1 for end-to-end, all or nothing for
//                 TPOT (F - P against thr * l_out, which does not depend on the start);
//                 0 when it can never be met, and past the last position.
// A move changes the members of at most two batches (A before C). Each is scored in one
// pass with its new members in lanes: a member that stays gets
//   F' = F + [pf(g) + w(g, m) / 2] - [pf(o) + w(o, m) / 2]
// for the request g that joins and o that leaves (either may be absent), and the newcomer
//   F'(g) = P' + L_g d0 + sum over the new members j of w(j, g) / 2,
// with w(j, m) = mu (e_j + d2 mu), mu = min(L_j, L_m), e_j = 2 (d1 + d2 l_j) + d2, twice
// what j adds to m's decode iterations. Four DPP reductions give P', the newcomer's sum,
// the new duration and the old one (the largest old offset of the members before the
// move), so that the start times of A and C before and after the move follow from one
// start read from the rows (swap: two). The two batches keep their members between them,
// so the change of t over them is a lane sum of new minus old latencies (old start: that
// of the old batch holding the member's old position). Later batches keep their members
// and only shift: by D'(A) - D(A) between A and C (swap), by the change of the end of the
// two batches after C. One pass over the register rows from A on writes the move's starts
// and limits and counts the change of the met flags by position: the positions of A and C
// lose their old flags (their new ones come from the batch passes), the shifted ones
// compare S + shift with lim. Most moves are accepted, so the rows are written before the
// decision and restored when the move is rejected; the order, layout and F change only
// on acceptance.
//
// Widths (checked on the device before any chain runs): every finish offset, batch
// prefill, doubled pair-cost sum over a batch and 24-bit multiply operand as in the
// fixed-size delta kernel, and every time on the timeline of any layout below 2^32 - 1.

struct SizedState {
  const uint4 *req;
  uint16_t *perm;
  uint8_t *flags;
  uint32_t *F;
  int n, B, lane;
  uint32_t d0, d2;
};

// f(integral_constant<int, u>) for u = 0 .. N-1: the row loops index their arrays with
// compile-time constants, so that each row becomes a register of its own (an array that
// the compiler keeps as one vector value is copied whole wherever an element changes)
template <class F, int... I>
__device__ __forceinline__ void static_for_seq(F &&f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, class F>
__device__ __forceinline__ void static_for(F &&f) {
  static_for_seq(f, std::make_integer_sequence<int, N>{});
}

// Rows of a wave's positions (S, lim) are plain register arrays indexed by constants only:
// the row of a single position is picked by a wave-uniform branch tree, so that every row
// keeps a register of its own.
template <int LO, int HI, int NR>
__device__ __forceinline__ uint32_t row_lane(const uint32_t (&v)[NR], int u, int l) {
  if constexpr (HI - LO == 1) {
    return readlane(v[LO], l);
  } else {
    constexpr int MID = (LO + HI) / 2;
    if (u < MID) return row_lane<LO, MID>(v, u, l);
    return row_lane<MID, HI>(v, u, l);
  }
}
template <int LO, int HI, int NR>
__device__ __forceinline__ void set_row_lane(uint32_t (&v)[NR], int u, int l, uint32_t x) {
  if constexpr (HI - LO == 1) {
    v[LO] = wlane_m0(x, l, v[LO]);
  } else {
    constexpr int MID = (LO + HI) / 2;
    if (u < MID)
      set_row_lane<LO, MID>(v, u, l, x);
    else
      set_row_lane<MID, HI>(v, u, l, x);
  }
}
// start of the batch holding position x (x < n)
template <int NR>
__device__ __forceinline__ uint32_t start_at(const uint32_t (&S)[NR], int x) {
  return row_lane<0, NR>(S, x >> 6, x & 63);
}
template <int NR>
__device__ __forceinline__ void swap_lims(uint32_t (&lim)[NR], int x, int y) {
  const uint32_t a = row_lane<0, NR>(lim, x >> 6, x & 63), b = row_lane<0, NR>(lim, y >> 6, y & 63);
  set_row_lane<0, NR>(lim, x >> 6, x & 63, b);
  set_row_lane<0, NR>(lim, y >> 6, y & 63, a);
}

// Number of register rows for n positions (the kernel is instantiated for these).
__host__ __device__ constexpr int sized_rows_for(int n) { return n <= 128 ? 2 : (n <= 256 ? 4 : (n <= 512 ? 8 : 16)); }

// limit of a member: met iff batch start < limit
// (both forms on every lane and a select: lanes of one wave hold requests of every kind)
__device__ __forceinline__ uint32_t member_limit(uint32_t kind, uint32_t thr, uint32_t P, uint32_t F) {
  const uint32_t off = kind == 0 ? P : F;
  const uint32_t by_start = thr >= off ? thr - off + 1u : 0u;
  const uint32_t tpot = F - P <= thr ? 0xFFFFFFFFu : 0u;
  return kind == 1 ? tpot : by_start;
}

// One changed batch [xs, xe) with its new members in lanes 0 .. xe - xs - 1 (lanes past
// the batch read its last member's records, or the first position's, and are masked out):
// what needs no start time -- each member's new finish offset and limit, its old offset
// and old position, the new duration and the old one (the members that stay and o, who
// leaves).
struct BatchNew {
  uint32_t Fn, limn, Fold;
  int r, q;
  bool act;
  uint32_t D, Dold, Pold;  // Pold: the old batch's prefill (the members before the move)
};

// Loads of one changed batch [xs, xe) (may be empty); the reductions follow in batch_scan2.
struct BatchLoad {
  Req rq, rg;
  uint32_t Fold, Fo, f, P, T, Mx, Mo, pfo;
  int r, q;
  bool act;
};
__device__ __forceinline__ BatchLoad batch_load(const SizedState &c, int xs, int xe, const Remap &rm, int g, int o) {
  const int p = xs + c.lane;
  const bool act = p < xe;
  const int q = rm.src(max(min(p, xe - 1), 0));
  const int r = c.perm[q];
  const Req rq = load_req(c.req, r);
  // absent g or o read the spare all-zero record: its prefill and pair costs vanish
  const Req rg = load_req(c.req, g >= 0 ? g : c.n), ro = load_req(c.req, o >= 0 ? o : c.n);
  const uint32_t Fold = c.F[r], Fo = o >= 0 ? c.F[max(o, 0)] : 0u;
  const uint32_t f = Fold + rg.pf + (w2(rg.L, rg.e, rq.L, c.d2) >> 1) - ro.pf - (w2(ro.L, ro.e, rq.L, c.d2) >> 1);
  const bool stay = act && r != g;
  return BatchLoad{rq, rg, Fold, Fo, f, act ? rq.pf : 0u, act ? w2(rq.L, rq.e, rg.L, c.d2) : 0u, stay ? f : 0u,
                   stay ? Fold : 0u, ro.pf, r, q, act};
}
__device__ __forceinline__ BatchNew batch_finish(const SizedState &c, const BatchLoad &l, int g) {
  const uint32_t Fg = g >= 0 ? l.P + __umul24(l.rg.L, c.d0) + (l.T >> 1) : 0u;
  const uint32_t Fn = l.r == g ? Fg : l.f;
  const uint32_t limn = member_limit(l.rq.kind, l.rq.thr, l.P, Fn);
  return BatchNew{Fn, limn, l.Fold, l.r, l.q, l.act, max(l.Mx, Fg), max(l.Mo, l.Fo), l.P - l.rg.pf + l.pfo};
}
// Both changed batches at once (A and C; either may be empty, its lanes all masked out:
// duration 0, old duration that of the one who left it, if any), the eight reductions
// interleaved.
__device__ __forceinline__ void batch_scan2(const SizedState &c, int as, int ae, int gA, int oA, int cs, int ce, int gC,
                                            int oC, const Remap &rm, BatchNew &nA, BatchNew &nC) {
  BatchLoad a = batch_load(c, as, ae, rm, gA, oA), b = batch_load(c, cs, ce, rm, gC, oC);
#pragma unroll
  for (int st = 0; st < Seg<6>::kSteps; ++st) {
    a.P = Seg<6>::template step<OpAdd>(a.P, st);
    b.P = Seg<6>::template step<OpAdd>(b.P, st);
    a.T = Seg<6>::template step<OpAdd>(a.T, st);
    b.T = Seg<6>::template step<OpAdd>(b.T, st);
    a.Mx = Seg<6>::template step<OpMax>(a.Mx, st);
    b.Mx = Seg<6>::template step<OpMax>(b.Mx, st);
    a.Mo = Seg<6>::template step<OpMax>(a.Mo, st);
    b.Mo = Seg<6>::template step<OpMax>(b.Mo, st);
  }
  a.P = readlane(a.P, kWave - 1), a.T = readlane(a.T, kWave - 1), a.Mx = readlane(a.Mx, kWave - 1);
  a.Mo = readlane(a.Mo, kWave - 1);
  b.P = readlane(b.P, kWave - 1), b.T = readlane(b.T, kWave - 1), b.Mx = readlane(b.Mx, kWave - 1);
  b.Mo = readlane(b.Mo, kWave - 1);
  nA = batch_finish(c, a, gA);
  nC = batch_finish(c, b, gC);
}

// The rest, with the batch's new start SX: adds to dt the change of its members'
// latencies (old start S0 for old positions before ob, S1 from ob on) and to the lane
// counter met whether the lane's member meets its SLO in the new batch.
__device__ __forceinline__ void batch_tally(const BatchNew &b, uint32_t SX, int ob, uint32_t S0, uint32_t S1,
                                            int64_t &dt, int &met) {
  met += (b.act && SX < b.limn) ? 1 : 0;
  const uint32_t Sold = b.q < ob ? S0 : S1;
  dt += b.act ? (int64_t)(SX + b.Fn) - (int64_t)(Sold + b.Fold) : 0;
}

// Rows by their place against the changed ranges: before r0 wholly before b0 (untouched),
// from rE on wholly at or after b3 (shifted by sE), in [rM0, rM1) wholly inside [b1, b2)
// (shifted by sM); the others hold positions of A or C or a range bound.
struct RowSpan {
  int r0, rE, rM0, rM1;
};
__device__ __forceinline__ RowSpan row_span(int b0, int b1, int b2, int b3) {
  return RowSpan{b0 >> 6, (b3 + kWave - 1) >> 6, (b1 + kWave - 1) >> 6, b2 >> 6};
}

// The move on the rows, before it is decided (most proposals that make a move are
// accepted; a rejected one is undone by row_undo): A = [b0, b1) takes start SA and limits
// limA (by lane position), C = [b2, b3) start SC and limits limC, [b1, b2) shifts by sM,
// [b3, n] by sE (b0 <= b1 <= b2 <= b3). Returns the lane's change of the met flags from b0
// on: the positions of A and C lose their old flags (their new ones are counted by the
// batch tallies), the shifted ones compare the new start with the limit. The lane index
// comes in as a fresh copy each call, so that no per-row position is kept live across
// calls.
template <int NR>
__device__ __forceinline__ int row_update(uint32_t (&S)[NR], uint32_t (&lim)[NR], int lane, int b0, int b1, int b2,
                                          int b3, uint32_t sM, uint32_t sE, uint32_t SA, uint32_t SC, uint32_t limA,
                                          uint32_t limC) {
  const RowSpan rs = row_span(b0, b1, b2, b3);
  int cnt = 0;
  static_for<NR>([=, &S, &lim, &cnt](auto uc) __attribute__((always_inline)) {
    constexpr int u = decltype(uc)::value;
    if (u < rs.r0) return;
    const uint32_t s = S[u], l = lim[u];
    // each branch forms its own contribution behind an opaque copy: merged, the branches
    // would leave a lane-mask merge through the exec mask after them
    int v;
    if (u >= rs.rE) {
      const uint32_t x = s + sE;
      v = (int)(x < l) - (int)(s < l);
      S[u] = x;
      asm volatile("" : "+v"(v));
    } else if (u >= rs.rM0 && u < rs.rM1) {
      const uint32_t x = s + sM;
      v = (int)(x < l) - (int)(s < l);
      S[u] = x;
      asm volatile("" : "+v"(v));
    } else {
      const int p = lane + u * kWave;
      const bool inA = (unsigned)(p - b0) < (unsigned)(b1 - b0), inC = (unsigned)(p - b2) < (unsigned)(b3 - b2);
      const uint32_t d = p >= b3 ? sE : (p >= b1 ? sM : 0u);
      const uint32_t x = s + d;
      v = (int)(!(inA || inC) && x < l) - (int)(s < l);
      uint32_t sn = inC ? SC : x;
      sn = inA ? SA : sn;
      uint32_t ln = inC ? limC : l;
      ln = inA ? limA : ln;
      S[u] = sn;
      lim[u] = ln;
      asm volatile("" : "+v"(v));
    }
    cnt += v;
  });
  return cnt;
}

// Undoes row_update for a rejected move: shifted positions move back, the positions of A
// and C take their old start (SA before ob, S1 from ob on) and their old limit, formed
// again from the order and offsets (both still the old ones) and the old batch prefills
// (PA before ob, PC from ob on).
template <int NR>
__device__ __forceinline__ void row_undo(const SizedState &c, uint32_t (&S)[NR], uint32_t (&lim)[NR], int lane, int b0,
                                         int b1, int b2, int b3, uint32_t sM, uint32_t sE, int ob, uint32_t SA,
                                         uint32_t S1, uint32_t PA, uint32_t PC) {
  const RowSpan rs = row_span(b0, b1, b2, b3);
  static_for<NR>([=, &S, &lim](auto uc) __attribute__((always_inline)) {
    constexpr int u = decltype(uc)::value;
    if (u < rs.r0) return;
    if (u >= rs.rE) {
      S[u] -= sE;
    } else if (u >= rs.rM0 && u < rs.rM1) {
      S[u] -= sM;
    } else {
      const int p = lane + u * kWave;
      const bool chg = (unsigned)(p - b0) < (unsigned)(b1 - b0) || (unsigned)(p - b2) < (unsigned)(b3 - b2);
      const uint32_t d = p >= b3 ? sE : (p >= b1 ? sM : 0u);
      const bool first = p < ob;
      const int r = c.perm[min(p, c.n - 1)];
      const Req rq = load_req(c.req, r);
      const uint32_t lo = member_limit(rq.kind, rq.thr, first ? PA : PC, c.F[r]);
      S[u] = chg ? (first ? SA : S1) : S[u] - d;
      lim[u] = chg ? lo : lim[u];
    }
  });
}

// F, S, lim of an order with maximum-size batches; returns its (n, t).
template <int NR>
__device__ __forceinline__ Score sized_init(const SizedState &c, uint32_t (&S)[NR], uint32_t (&lim)[NR]) {
  const int lane = c.lane;
  // an opaque zero: stores of a constant would be merged into one block fill, after which
  // the compiler keeps the rows as one vector value
  uint32_t zero = 0u;
  asm volatile("" : "+v"(zero));
  static_for<NR>([&S, &lim, zero](auto uc) __attribute__((always_inline)) {
    S[decltype(uc)::value] = zero;
    lim[decltype(uc)::value] = zero;
  });
  uint32_t Sc = 0;
  int64_t nmet = 0;
  uint64_t tl = 0;
  for (int s = 0; s < c.n; s += c.B) {
    const int b = min(c.B, c.n - s);
    const bool act = lane < b;
    const int r = act ? (int)c.perm[s + lane] : c.n;
    const Req rq = load_req(c.req, r);
    uint32_t acc = 0;
    for (int j = 0; j < b; ++j) {
      const uint32_t Lj = readlane(rq.L, j), ej = readlane(rq.e, j);
      acc += w2(Lj, ej, rq.L, c.d2);
    }
    uint32_t P = act ? rq.pf : 0u;
    P = Seg<6>::template all<OpAdd>(P, lane);
    const uint32_t F = act ? P + __umul24(rq.L, c.d0) + (acc >> 1) : 0u;
    const uint32_t D = Seg<6>::template all<OpMax>(F, lane);
    const uint32_t limv = member_limit(rq.kind, rq.thr, P, F);
    if (act) {
      c.F[r] = F;
      tl += (uint64_t)(Sc + F);
    }
    nmet += __popcll(__ballot(act && Sc < limv));
    // lane l holds position s + l: rotate into the rows' lanes
    const uint32_t lr = (uint32_t)__shfl((int)limv, (lane - s) & 63);
    static_for<NR>([=, &S, &lim](auto uc) __attribute__((always_inline)) {
      constexpr int u = decltype(uc)::value;
      const bool mine = (unsigned)(u * kWave + lane - s) < (unsigned)b;
      S[u] = mine ? Sc : S[u];
      lim[u] = mine ? lr : lim[u];
    });
    Sc += D;
  }
  wave_sync_lds();
  return Score{nmet, wave_sum_u64(tl)};
}

// One wave per chain, blockDim / 64 chains per workgroup, positions in NR register rows
// (n <= 64 NR).
template <int OBJ, int NR>
__global__ void __launch_bounds__(1024) anneal_sized_kernel(DevModel m, StaticParams sp, QueuePtrs q, int chains,
                                                             int iters, double T0, double alpha, uint32_t key0,
                                                             uint32_t key1, SearchParams srch, unsigned char *ws) {
  extern __shared__ __align__(16) unsigned char lds[];
  if (!gate_open(ws, m.gate, m.flags)) return;
  const int n = m.n, B = m.B;
  const int waves = blockDim.x >> 6;
  uint4 *req = reinterpret_cast<uint4 *>(lds);
  const size_t pb = ((size_t)n * 2 + 15) & ~size_t(15), fb = ((size_t)n + 15) & ~size_t(15);
  const size_t ub = ((size_t)n * 4 + 15) & ~size_t(15);
  const size_t per_wave = pb + fb + ub;
  const int wave = uniform((int)(threadIdx.x >> 6));
  unsigned char *wb = lds + (size_t)(n + 1) * 16 + (size_t)wave * per_wave;
  for (int r = threadIdx.x; r <= n; r += blockDim.x) {
    if (r == n) {
      req[r] = make_uint4(0u, 0u, 0u, 0u);  // spare record: a zero request for absent movers
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
  const int chain = uniform((int)blockIdx.x * waves + wave);
  if (chain >= chains) return;
  const int lane = lane_id();
  SizedState c{req,
               reinterpret_cast<uint16_t *>(wb),
               wb + pb,
               reinterpret_cast<uint32_t *>(wb + pb + fb),
               n, B, lane, sp.d0, sp.d2};
  uint32_t S[NR], lim[NR];  // register rows (position p: row p / 64, lane p % 64)
  const WsHeader *h = reinterpret_cast<const WsHeader *>(ws);
  const int64_t t_ref = h->t_ref, allmet = h->allmet;
  const uint16_t *start = reinterpret_cast<const uint16_t *>(ws + ws_off_start());
  const size_t stride = ws_perm_stride(n), fstride = ws_flag_stride(n);
  uint16_t *gbest = reinterpret_cast<uint16_t *>(ws + ws_off_best(n, chains)) + (size_t)chain * stride;
  uint16_t *gcur = reinterpret_cast<uint16_t *>(ws + ws_off_cur(n, chains)) + (size_t)chain * stride;
  uint8_t *gbest_f = ws + ws_off_best_starts(n, chains) + (size_t)chain * fstride;
  uint8_t *gcur_f = ws + ws_off_cur_starts(n, chains) + (size_t)chain * fstride;
  for (int p = lane; p < n; p += kWave) {
    const uint16_t v = start[p];
    const uint8_t fl = (uint8_t)(p % B == 0);
    c.perm[p] = v;
    c.flags[p] = fl;
    gbest[p] = v;
    gbest_f[p] = fl;
  }
  wave_sync_lds();
  const Score s0 = sized_init(c, S, lim);
  int64_t cn = s0.n, bn = s0.n, biter = -1, accepts = 0;
  uint64_t ct = s0.t, bt = s0.t, digest = kFnvOffset;
  Cooling cool{T0, alpha, srch.level_len, srch.level_len};
  SizedDraws ds;
  const int iters_run = (srch.early_exit && allmet) ? 0 : iters;
  for (int k = 0; k < iters_run; ++k) {
    if ((k & (kWave - 1)) == 0) ds.refill(k, lane, n, (uint32_t)chain, key0, key1);
    const uint32_t pk = ds.packed(k), w3 = ds.word3(k);
    const int op = (int)(pk >> 20), i = (int)(pk & 1023u), j = (int)((pk >> 10) & 1023u);
    // plan: new ranges of the changed batches A = [as, ae) and C = [cs, ce), who joins and
    // leaves each, the range between them (swap) and the flag writes. Old positions
    // before ob belonged to a batch starting at SA, the others to one starting at S1. The
    // start times come from the register rows at the positions xa (swap: also xc), in the
    // old batch of A (in_first) or the second old batch, and the old durations of the
    // batches from the scans.
    bool made = false, inside = false, in_first = true;
    int as = 0, ae = 0, cs = 0, ce = 0, gA = -1, oA = -1, gC = -1, oC = -1, ob = n, xa = 0, xc = 0, x = 0;
    int set0 = -1, clr0 = -1;
    Remap rm{0, 0, 0};
    if (op == 2) {
      if (n >= 2) {
        made = true;
        const int lo = min(i, j), hi = max(i, j);
        const int sa = batch_begin(c.flags, lo, lane), ea = batch_end(c.flags, n, lo, lane);
        rm = Remap{1, lo, hi};
        if (hi < ea) {
          inside = true;
        } else {
          const int sc = batch_begin(c.flags, hi, lane), ec = batch_end(c.flags, n, hi, lane);
          const int plo = uniform(c.perm[lo]), phi = uniform(c.perm[hi]);
          as = sa, ae = ea, cs = sc, ce = ec;
          gA = phi, oA = plo, gC = plo, oC = phi;
          ob = sc;
          xa = lo, xc = hi;
        }
      }
    } else {
      const int s = batch_begin(c.flags, i, lane), e = batch_end(c.flags, n, i, lane);
      x = uniform(c.perm[i]);
      xa = i;
      if (op == 0) {
        if (s > 0) {
          const int sp2 = batch_begin(c.flags, s - 1, lane);
          if (s - sp2 < B) {
            made = true;
            rm = Remap{2, i, s};
            as = sp2, ae = s + 1, gA = x;
            cs = s + 1, ce = e, oC = x;
            clr0 = s;
            set0 = s + 1 < e ? s + 1 : -1;
            ob = s;
            in_first = false;
          }
        }
      } else if (e == n) {
        if (e - s >= 2) {
          made = true;
          rm = Remap{2, i, n - 1};
          as = s, ae = n - 1, oA = x;
          cs = n - 1, ce = n, gC = x;
          set0 = n - 1;
        }
      } else {
        const int en = batch_end(c.flags, n, e, lane);
        if (en - e < B) {
          made = true;
          rm = Remap{2, i, e - 1};
          as = s, ae = e - 1, oA = x;
          cs = e - 1, ce = en, gC = x;
          set0 = e - 1;
          clr0 = e;
          ob = e;
        }
      }
    }
    if (!made) {
      cool.step();
      continue;
    }
    int64_t dT = 0;
    int dn = 0;
    BatchNew nA{}, nC{};
    uint32_t SA = 0, SC = 0, S1k = 0, shift_mid = 0, shift_end = 0;
    if (!inside) {
      const uint32_t Sa = start_at(S, xa), Sc = op == 2 ? start_at(S, xc) : 0u;
      batch_scan2(c, as, ae, gA, oA, cs, ce, gC, oC, rm, nA, nC);
      const uint32_t DA = nA.D, DAold = nA.Dold, DC = nC.D, DCold = nC.Dold;
      // old starts: SA of the old batch of A, S1 of the second old batch
      uint32_t S1;
      if (op == 2) {
        SA = Sa;
        S1 = Sc;
        SC = S1 + DA - DAold;
      } else {
        SA = in_first ? Sa : Sa - DAold;
        S1 = in_first ? Sa + DAold : Sa;
        SC = SA + DA;
      }
      int64_t dtl = 0;
      int met = 0;
      batch_tally(nA, SA, ob, SA, S1, dtl, met);
      batch_tally(nC, SC, ob, SA, S1, dtl, met);
      // end of the two batches before the move (an insert that opens a new last batch:
      // S1 is the end of the only old batch and C had no old members)
      const uint32_t old_end = S1 + DCold;
      shift_end = SC + DC - old_end;
      shift_mid = DA - DAold;  // used between A and C of a swap only
      // the new limits of A and C, lane l of a batch scan holding position start + l,
      // rotated into the rows' lanes
      const uint32_t limA = (uint32_t)__shfl((int)nA.limn, (lane - as) & 63);
      const uint32_t limC = (uint32_t)__shfl((int)nC.limn, (lane - cs) & 63);
      int lnr = lane;
      asm volatile("" : "+v"(lnr));
      met += row_update(S, lim, lnr, as, ae, cs, ce, shift_mid, shift_end, SA, SC, limA, limC);
      S1k = S1;
      // one reduction for the met count and the latency change, the latter as two exact
      // parts (each lane's change lies within +-2^33: 2^24 * sum(hi) + sum(lo))
      uint32_t mu = (uint32_t)met, lo = (uint32_t)dtl & 0xFFFFFFu, hi = (uint32_t)(int32_t)(dtl >> 24);
      Seg<6>::template all3<OpAdd, OpAdd, OpAdd>(mu, lo, hi, lane);
      dn = (int)mu;
      dT = ((int64_t)(SC + DC) - (int64_t)old_end) * (int64_t)(n - ce);
      if (op == 2) dT += ((int64_t)DA - (int64_t)DAold) * (int64_t)(cs - ae);
      dT += (int64_t)(int32_t)hi * (int64_t)(1 << 24) + (int64_t)lo;
    }
    const int64_t nn = cn + dn;
    const uint64_t nt = ct + (uint64_t)dT;
    if (obj_accept<OBJ>(cn, ct, dn, dT, t_ref, cool.T, w3)) {
      if (inside) {
        swap_lims(lim, rm.i, rm.j);
        apply_move_lds(c.perm, 1, rm.i, rm.j, lane);
      } else {
        apply_move_lds(c.perm, rm.kind, rm.i, rm.j, lane);
        if (lane == 0) {
          if (clr0 >= 0) c.flags[clr0] = 0;
          if (set0 >= 0) c.flags[set0] = 1;
        }
        if (as + lane < ae) c.F[nA.r] = nA.Fn;
        if (cs + lane < ce) c.F[nC.r] = nC.Fn;
        wave_sync_lds();
      }
      cn = nn;
      ct = nt;
      ++accepts;
      digest = (digest ^ (uint64_t)k) * kFnvPrime;
      digest = (digest ^ (uint64_t)cn) * kFnvPrime;
      digest = (digest ^ ct) * kFnvPrime;
      if (obj_better<OBJ>(cn, ct, bn, bt)) {
        bn = cn;
        bt = ct;
        biter = k;
        for (int p = lane; p < n; p += kWave) {
          gbest[p] = c.perm[p];
          gbest_f[p] = c.flags[p];
        }
      }
    } else if (!inside) {
      int lnu = lane;
      asm volatile("" : "+v"(lnu));
      row_undo(c, S, lim, lnu, as, ae, cs, ce, shift_mid, shift_end, ob, SA, S1k, nA.Pold, nC.Pold);
    }
    cool.step();
  }
  for (int p = lane; p < n; p += kWave) {
    gcur[p] = c.perm[p];
    gcur_f[p] = c.flags[p];
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
