// Several serving instances (gfx950, wave64): the instance assignment of the Scheduling
// Solution (Algorithm 2's InstAssign) and the priority mapping of every instance in one
// launch per step.
//
// Assignment: requests in arrival order, each to the instance with the largest remaining
// memory in tokens (the caller's capacities, token_num(m) = m mu / sigma); when even that
// instance cannot hold the request (l_in + l_out tokens), every instance is reset to its
// capacity -- a fresh iteration -- and the request goes to the roomiest one. Ties go to the
// lowest index. One wave: lane k holds instance k's remaining tokens, and each request is
// one wave argmax.
//
// Per-instance annealing: instance k's requests, in arrival order, form its own queue; its
// chain c is the single-queue chain on that queue drawing from Philox chain index
// k * chains + c. Every step is one launch over all instances: the gather (one workgroup per
// instance), the start orders (one workgroup per instance), the chains (instances x chain
// groups, one wave per chain, full replay per proposal) and the winners (one workgroup per
// instance). The paper runs the instances one after another; here they run side by side.
//
// Workspace: a 256-byte header (n, instances, chains, slot size), a table of 64 bytes per
// instance (its request count), then one slot per instance: a single-queue workspace laid
// out for the instance's request count (so the single-queue readouts work on it), followed
// by the instance's queue (structure of arrays) and the global ids of its requests.
#pragma once
#include "anneal_reg.h"
#include "anneal_static.h"
#include "anneal_wave.h"
#include "kernels.h"

namespace sa {

constexpr uint64_t kMultiMagic = 0x534c4f4d554c5431ull;  // "SLOMULT1"

struct MultiHeader {
  uint64_t magic;
  int32_t n, instances, chains, pad;
  int64_t slot_bytes;
  int64_t reserved0[10];
  // the device checks' verdict, at the offsets a single-queue header keeps it
  int64_t plan_status, plan_flags, plan_selected;
  int64_t reserved[15];
};
static_assert(sizeof(MultiHeader) <= 256, "header fits its slot");
static_assert(offsetof(MultiHeader, plan_status) == offsetof(WsHeader, plan_status) &&
                  offsetof(MultiHeader, plan_flags) == offsetof(WsHeader, plan_flags) &&
                  offsetof(MultiHeader, plan_selected) == offsetof(WsHeader, plan_selected),
              "the verdict sits where the single-queue readers look");

__host__ __device__ __forceinline__ size_t mws_queue_bytes(int n) {
  const size_t a = round_up((size_t)n * 2, 256), b = round_up((size_t)n, 256), c = round_up((size_t)n * 4, 256);
  return 3 * a + b + c;  // in_len, out_len, ids (u16); kind (u8); thr (u32)
}
__host__ __device__ __forceinline__ size_t mws_slot_bytes(int n, int chains) {
  return round_up(ws_total(n, chains), 256) + mws_queue_bytes(n);
}
__host__ __device__ __forceinline__ size_t mws_off_table() { return 256; }
__host__ __device__ __forceinline__ size_t mws_off_slot(int n, int instances, int chains, int k) {
  return 256 + round_up((size_t)instances * 64, 256) + (size_t)k * mws_slot_bytes(n, chains);
}
__host__ __device__ __forceinline__ size_t mws_total(int n, int instances, int chains) {
  return mws_off_slot(n, instances, chains, instances);
}

// The instance's queue inside its slot.
struct SlotQueue {
  uint16_t *in_len, *out_len, *ids;
  uint8_t *kind;
  uint32_t *thr;
};
__host__ __device__ __forceinline__ SlotQueue slot_queue(unsigned char *slot, int n, int chains) {
  unsigned char *base = slot + round_up(ws_total(n, chains), 256);
  const size_t a = round_up((size_t)n * 2, 256), b = round_up((size_t)n, 256);
  return SlotQueue{reinterpret_cast<uint16_t *>(base), reinterpret_cast<uint16_t *>(base + a),
                   reinterpret_cast<uint16_t *>(base + 2 * a), base + 3 * a,
                   reinterpret_cast<uint32_t *>(base + 3 * a + b)};
}

// Capacities below this many tokens take the sorted-key assignment below.
constexpr int64_t kAssignNarrowCap = int64_t(1) << 25;

// One wave: instance of every request, every capacity below kAssignNarrowCap. Instance k's
// remaining tokens rem travel in a 32-bit key ((rem + 2^17) << 6) | (63 - k): rem stays
// above -2^17 (an instance is overdrawn only by the first request after a reset, by less
// than one request of at most 2 * 65535 tokens) and below 2^25, so the key is positive and
// below 2^32, larger keys mean more room, and equal room orders the lower index first.
// The keys sit in lanes sorted in descending order (lanes past the instances hold 0), so
// the roomiest instance is lane 0; placing a request pops it and inserts the reduced key,
// and lane i of the new list is the median of list[i], list[i + 1] and that key (one DPP
// shift and one v_med3_u32). A reset restores the initial sorted list. Request sizes are
// loaded 64 at a time and the instances written 64 at a time.
__device__ __forceinline__ void assign_sorted_body(const QueuePtrs &q, int n, int instances,
                                                   const int64_t *__restrict__ capacity,
                                                   int32_t *__restrict__ inst_out) {
  __shared__ uint32_t srt[64];
  const int lane = lane_id();
  const bool live = lane < instances;
  const uint32_t key0 = live ? ((uint32_t)(capacity[lane] + (int64_t(1) << 17)) << 6) | (uint32_t)(63 - lane) : 0u;
  // rank among the instances' keys (distinct by their index bits); other lanes keep theirs
  int rank = lane;
  if (live) {
    rank = 0;
    for (int u = 0; u < instances; ++u) rank += (uint32_t)__builtin_amdgcn_readlane((int)key0, u) > key0 ? 1 : 0;
  }
  srt[rank] = key0;
  __syncthreads();
  const uint32_t init = srt[lane];
  const uint32_t init_top = (uint32_t)__builtin_amdgcn_readfirstlane((int)init);
  uint32_t list = init;
  for (int c0 = 0; c0 < n; c0 += kWave) {
    const int cnt = min(kWave, n - c0);
    const uint32_t needv = lane < cnt ? (uint32_t)q.in_len[c0 + lane] + (uint32_t)q.out_len[c0 + lane] : 0u;
    uint32_t outv = 0;
    for (int t = 0; t < cnt; ++t) {
      const uint32_t need = (uint32_t)__builtin_amdgcn_readlane((int)needv, t);
      uint32_t top = (uint32_t)__builtin_amdgcn_readfirstlane((int)list);
      if ((int32_t)(top >> 6) - (1 << 17) < (int32_t)need) {  // even the roomiest cannot hold it
        list = init;
        top = init_top;
      }
      const uint32_t nk = top - (need << 6);
      const uint32_t above = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)list, 0x130, 0xF, 0xF, true);  // list[i + 1]
      list = med3_u32(above, list, nk);
      const uint32_t k = 63u - (top & 63u);
      outv = lane == t ? k : outv;
    }
    if (lane < cnt) inst_out[c0 + lane] = (int32_t)outv;
  }
}

// One wave: instance of every request, 64-bit remaining tokens (any capacity).
__device__ __forceinline__ void assign_wide_body(const QueuePtrs &q, int n, int instances,
                                                 const int64_t *__restrict__ capacity, int32_t *__restrict__ inst_out) {
  const int lane = lane_id();
  const bool live = lane < instances;
  const int64_t cap = live ? capacity[lane] : INT64_MIN;
  int64_t rem = cap;
  // the roomiest instance at a reset: largest capacity, lowest index
  auto argmax = [lane](int64_t v) {
    int64_t bv = v;
    int bk = lane;
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
      const int64_t ov = __shfl_xor(bv, o);
      const int ok = __shfl_xor(bk, o);
      if (ov > bv || (ov == bv && ok < bk)) {
        bv = ov;
        bk = ok;
      }
    }
    return bk;
  };
  const int kcap = uniform(argmax(cap));
  for (int r = 0; r < n; ++r) {
    const int64_t need = (int64_t)q.in_len[r] + (int64_t)q.out_len[r];
    int k = uniform(argmax(rem));
    const int64_t best_rem = __shfl(rem, k);
    if (best_rem < need) {
      rem = cap;
      k = kcap;
    }
    if (lane == k) rem -= need;
    if (lane == 0) inst_out[r] = k;
  }
}

// One wave: the checks of the assignment (every queue entry as for the other calls, every
// capacity within 1 .. 2^48; on failure every entry of inst_out reads SCHED_EINVAL), then
// the sorted-key body when every capacity is below kAssignNarrowCap, else the 64-bit one.
__global__ void __launch_bounds__(64) assign_kernel(QueuePtrs q, int n, int instances,
                                                     const int64_t *__restrict__ capacity, int32_t *__restrict__ inst_out) {
  const int lane = lane_id();
  bool bad = false, wide = false;
  for (int r = lane; r < n; r += kWave)
    bad |= q.out_len[r] < 1u || q.kind[r] > 2u || q.thr[r] > kThrMax;
  if (lane < instances) {
    const int64_t c = capacity[lane];
    bad |= c < 1 || c > (int64_t(1) << 48);
    wide = c >= kAssignNarrowCap;
  }
  if (__ballot(bad) != 0ull) {
    for (int r = lane; r < n; r += kWave) inst_out[r] = kPlanEInval;
    return;
  }
  if (__ballot(wide) == 0ull)
    assign_sorted_body(q, n, instances, capacity, inst_out);
  else
    assign_wide_body(q, n, instances, capacity, inst_out);
}

// One workgroup of 1024 threads: the device checks of a several-instance call -- every queue
// entry, every instance index within 0 .. instances - 1, the int64 range and widths of the
// whole queue (each instance's queue is part of it, so its bounds hold there too) and each
// instance's request count (at most 64 or 192 requests: the register kernels) -- and the
// multi-instance header; every slot's header gets the verdict too, so that the single-queue
// readouts on a slot see it.
__global__ void __launch_bounds__(1024) multi_plan_kernel(DevModel m, QueuePtrs q, const int32_t *__restrict__ inst_of,
                                                           int instances, int chains, int iters, int64_t slot_bytes,
                                                           unsigned char *mws) {
  __shared__ int cnt[64];
  __shared__ uint32_t bad_inst;
  const int n = m.n;
  if (threadIdx.x < 64) cnt[threadIdx.x] = 0;
  if (threadIdx.x == 0) bad_inst = 0u;
  __syncthreads();
  for (int r = threadIdx.x; r < n; r += blockDim.x) {
    const int32_t k = inst_of[r];
    if (k < 0 || k >= instances)
      atomicOr(&bad_inst, 1u);
    else
      atomicAdd(&cnt[k], 1);
  }
  QueueStats s = block_queue_stats(q, n, m.B, m.max_kind, nullptr);  // its barrier orders the counts
  s.bad |= bad_inst;
  int nk_max = 0;
  for (int k = 0; k < instances; ++k) nk_max = max(nk_max, cnt[k]);
  Plan p = plan_decide(s, n, m.B, m.ratio, m.t_ref, m.p0, m.p1, m.d0, m.d1, m.d2, nullptr, m.gate);
  if (p.status == 0) {
    if (nk_max <= 64) p.flags |= kFlagInst64;
    if (nk_max <= 192) p.flags |= kFlagInst192;
    p.selected = plan_select(m.gate, p.flags);
  }
  if (threadIdx.x == 0) {
    MultiHeader *mh = reinterpret_cast<MultiHeader *>(mws);
    mh->magic = kMultiMagic;
    mh->n = n;
    mh->instances = instances;
    mh->chains = chains;
    mh->slot_bytes = slot_bytes;
    mh->plan_status = p.status;
    mh->plan_flags = p.flags;
    mh->plan_selected = p.selected;
  }
  if ((int)threadIdx.x < instances) {
    unsigned char *slot = mws + mws_off_slot(n, instances, chains, (int)threadIdx.x);
    if (p.status != 0)
      write_failed_header(slot, p, 0, chains, iters, m.policy, m.B);
    else
      write_plan(slot, p);
  }
}

// One workgroup of 1024 threads per instance: the instance's requests in arrival order.
__global__ void __launch_bounds__(1024) gather_kernel(QueuePtrs q, int n, const int32_t *__restrict__ inst_of, int chains,
                                                       int instances, unsigned char *mws) {
  __shared__ int wave_cnt[16];
  if (!plan_ok(mws)) return;
  const int k = blockIdx.x;
  const int tid = threadIdx.x, lane = lane_id(), wave = tid >> 6;
  const bool mine = tid < n && inst_of[tid] == k;
  const uint64_t bal = __ballot(mine);
  if (lane == 0) wave_cnt[wave] = __popcll(bal);
  __syncthreads();
  int before = 0, total = 0;
  for (int w = 0; w < (int)(blockDim.x >> 6); ++w) {
    before += w < wave ? wave_cnt[w] : 0;
    total += wave_cnt[w];
  }
  unsigned char *slot = mws + mws_off_slot(n, instances, chains, k);
  const SlotQueue sq = slot_queue(slot, n, chains);
  if (mine) {
    const int p = before + rank_in_mask(bal);
    sq.in_len[p] = q.in_len[tid];
    sq.out_len[p] = q.out_len[tid];
    sq.kind[p] = q.kind[tid];
    sq.thr[p] = q.thr[tid];
    sq.ids[p] = (uint16_t)tid;
  }
  if (tid == 0) reinterpret_cast<int64_t *>(mws + mws_off_table())[8 * k] = total;
}

__device__ __forceinline__ int slot_n(const unsigned char *mws, int k) {
  return (int)reinterpret_cast<const int64_t *>(mws + mws_off_table())[8 * k];
}

// One workgroup per instance: its start order and workspace header.
__global__ void __launch_bounds__(1024) multi_start_kernel(DevModel m, int n, int instances, int chains, int iters,
                                                            int64_t t_ref_user, SearchParams srch, unsigned char *mws) {
  if (!gate_status(mws, m.gate, m.flags)) return;
  const int k = blockIdx.x;
  const int nk = slot_n(mws, k);
  unsigned char *slot = mws + mws_off_slot(n, instances, chains, k);
  if (nk == 0) {
    if (threadIdx.x == 0) {
      WsHeader *h = reinterpret_cast<WsHeader *>(slot);
      h->magic = kWsMagic;
      h->n = 0;
      h->chains = chains;
      h->iters = iters;
      h->policy = m.policy;
      h->max_batch = m.B;
      h->objective = srch.objective;
      h->level_len = srch.level_len;
      h->early_exit = srch.early_exit;
      h->t_ref = 1;
      h->start_n = 0;
      h->start_t = 0;
      h->allmet = 1;
      h->best_chain = -1;
      h->best_n = -1;
      h->best_t = -1;
    }
    return;
  }
  const SlotQueue sq = slot_queue(slot, n, chains);
  DevModel mk = m;
  mk.n = nk;
  start_body(mk, QueuePtrs{sq.in_len, sq.out_len, sq.kind, sq.thr}, chains, iters, t_ref_user, srch, slot);
}

// Instances x groups of 4 chains: one wave per chain, full replay per proposal. LDS is sized
// by the host for the largest instance.
template <int OBJ>
__global__ void __launch_bounds__(kBlock) multi_anneal_kernel(DevModel m, int n, int instances, int chains, int groups,
                                                               int iters, double T0, double alpha, uint32_t key0,
                                                               uint32_t key1, uint64_t swap_thr, SearchParams srch,
                                                               unsigned char *mws) {
  extern __shared__ __align__(16) unsigned char lds[];
  if (!gate_open(mws, m.gate, m.flags)) return;
  const int k = blockIdx.x / groups, g = blockIdx.x - k * groups;
  const int nk = slot_n(mws, k);
  if (nk == 0) return;
  unsigned char *slot = mws + mws_off_slot(n, instances, chains, k);
  const SlotQueue sq = slot_queue(slot, n, chains);
  DevModel mk = m;
  mk.n = nk;
  uint4 *req = reinterpret_cast<uint4 *>(lds);
  const size_t per_wave = lds_align((size_t)nk * 2) * 2 + 64 * 16;
  const int wave = uniform((int)(threadIdx.x >> 6));
  unsigned char *wbase = lds + lds_align((size_t)nk * 16) + (size_t)wave * per_wave;
  load_requests(QueuePtrs{sq.in_len, sq.out_len, sq.kind, sq.thr}, mk, req);
  __syncthreads();
  const int chain = uniform(g * kWavesPerBlock + wave);
  if (chain >= chains) return;
  anneal_chain_body<OBJ>(mk, req, wbase, chains, chain, (uint32_t)(k * chains + chain), iters, T0, alpha, key0, key1,
                         swap_thr, srch, slot);
}

// Static admission with the delta kernels: instances x groups of `waves` chains, one wave per
// chain; LG = log2 of the batch lanes' group width (0..5: the row kernel) or 6 (one batch per
// wave). LDS is sized by the host for the largest instance; each workgroup lays it out for
// its own instance's request count.
template <int LG, int OBJ>
__global__ void __launch_bounds__(1024) multi_static_kernel(DevModel m, StaticParams sp, int n, int instances,
                                                             int chains, int groups, int iters, double T0,
                                                             double alpha, uint32_t key0, uint32_t key1,
                                                             uint64_t swap_thr, SearchParams srch, unsigned char *mws) {
  extern __shared__ __align__(16) unsigned char lds[];
  if (!gate_open(mws, m.gate, m.flags)) return;
  const int k = blockIdx.x / groups, g = blockIdx.x - k * groups;
  const int nk = slot_n(mws, k);
  if (nk == 0) return;
  unsigned char *slot = mws + mws_off_slot(n, instances, chains, k);
  const SlotQueue sq = slot_queue(slot, n, chains);
  DevModel mk = m;
  mk.n = nk;
  uint4 *req = reinterpret_cast<uint4 *>(lds);
  const int waves = blockDim.x >> 6;
  const int wave = uniform((int)(threadIdx.x >> 6));
  const size_t per = LG == 6 ? wave_chain_bytes(nk, m.B) : static_chain_bytes(nk, m.B);
  unsigned char *wb = lds + (size_t)(nk + 1) * 16 + (size_t)wave * per;
  load_static_records(QueuePtrs{sq.in_len, sq.out_len, sq.kind, sq.thr}, mk, req);
  __syncthreads();
  const int chain = uniform(g * waves + wave);
  if (chain >= chains) return;
  const uint32_t rng_chain = (uint32_t)(k * chains + chain);
  if constexpr (LG == 6)
    anneal_wave_body<OBJ>(mk, sp, req, wb, chains, chain, rng_chain, iters, T0, alpha, key0, key1, swap_thr, srch,
                          slot);
  else
    anneal_static_body<LG, OBJ>(mk, sp, req, wb, chains, chain, rng_chain, iters, T0, alpha, key0, key1, swap_thr,
                                srch, slot);
}

// Static admission on instances of at most 64 requests and batches of 1, 2, 4, 8 or 16: the
// register kernel's chain body per instance (block k / groups), no LDS.
template <int LG, int OBJ>
__global__ void __launch_bounds__(256) multi_reg_kernel(DevModel m, int n, int instances, int chains, int groups,
                                                         int iters, double T0, double alpha, uint32_t key0,
                                                         uint32_t key1, uint64_t swap_thr, SearchParams srch,
                                                         unsigned char *mws) {
  if (!gate_open(mws, m.gate, m.flags)) return;
  const int k = blockIdx.x / groups, g = blockIdx.x - k * groups;
  const int nk = slot_n(mws, k);
  if (nk == 0) return;
  const int waves = blockDim.x >> 6;
  const int chain = uniform(g * waves + (int)(threadIdx.x >> 6));
  if (chain >= chains) return;
  unsigned char *slot = mws + mws_off_slot(n, instances, chains, k);
  const SlotQueue sq = slot_queue(slot, n, chains);
  DevModel mk = m;
  mk.n = nk;
  const QueuePtrs qk{sq.in_len, sq.out_len, sq.kind, sq.thr};
  if (m.flags & kFlagTime32)
    anneal_reg_body<LG, OBJ, true>(mk, qk, chains, chain, (uint32_t)(k * chains + chain), iters, T0, alpha, key0, key1,
                                   swap_thr, srch, slot);
  else
    anneal_reg_body<LG, OBJ, false>(mk, qk, chains, chain, (uint32_t)(k * chains + chain), iters, T0, alpha, key0, key1,
                                    swap_thr, srch, slot);
}

// The same for instances of up to 192 requests (one, two or three positions per lane, by
// each instance's own request count).
template <int LG, int OBJ>
__global__ void __launch_bounds__(256) multi_reg_h_kernel(DevModel m, int n, int instances, int chains, int groups,
                                                           int iters, double T0, double alpha, uint32_t key0,
                                                           uint32_t key1, uint64_t swap_thr, SearchParams srch,
                                                           unsigned char *mws) {
  if (!gate_open(mws, m.gate, m.flags)) return;
  const int k = blockIdx.x / groups, g = blockIdx.x - k * groups;
  const int nk = slot_n(mws, k);
  if (nk == 0) return;
  const int waves = blockDim.x >> 6;
  const int chain = uniform(g * waves + (int)(threadIdx.x >> 6));
  if (chain >= chains) return;
  unsigned char *slot = mws + mws_off_slot(n, instances, chains, k);
  const SlotQueue sq = slot_queue(slot, n, chains);
  DevModel mk = m;
  mk.n = nk;
  anneal_reg_any<LG, OBJ>(mk, QueuePtrs{sq.in_len, sq.out_len, sq.kind, sq.thr}, chains, chain,
                          (uint32_t)(k * chains + chain), iters, T0, alpha, key0, key1, swap_thr, srch, slot);
}

// One workgroup per instance: its winner over chains.
__global__ void __launch_bounds__(1024) multi_reduce_kernel(int n, int instances, int chains, unsigned char *mws) {
  if (!plan_ok(mws)) return;
  const int k = blockIdx.x;
  if (slot_n(mws, k) == 0) return;
  reduce_body(mws + mws_off_slot(n, instances, chains, k));
}

// One workgroup per instance: its best order as global request ids, at the offset of the
// instance's first request in instance order; its key and request count.
__global__ void __launch_bounds__(256) multi_best_kernel(const unsigned char *mws, uint16_t *orders, int64_t *keys,
                                                          int32_t *counts) {
  const MultiHeader *mh = reinterpret_cast<const MultiHeader *>(mws);
  const int n = mh->n, instances = mh->instances, chains = mh->chains;
  const int k = blockIdx.x;
  if (mh->plan_status != 0) {  // the queue failed the checks: (-2, code, -1), no requests
    if (threadIdx.x == 0) {
      if (keys) {
        keys[3 * k] = -2;
        keys[3 * k + 1] = mh->plan_status;
        keys[3 * k + 2] = -1;
      }
      if (counts) counts[k] = 0;
    }
    return;
  }
  int off = 0;
  for (int j = 0; j < k; ++j) off += slot_n(mws, j);
  const int nk = slot_n(mws, k);
  const unsigned char *slot = mws + mws_off_slot(n, instances, chains, k);
  const WsHeader *h = reinterpret_cast<const WsHeader *>(slot);
  if (nk > 0) {
    const SlotQueue sq = slot_queue(const_cast<unsigned char *>(slot), n, chains);
    const int64_t c = h->best_chain;
    const uint16_t *best =
        reinterpret_cast<const uint16_t *>(slot + ws_off_best(nk, chains)) + (size_t)c * ws_perm_stride(nk);
    for (int p = threadIdx.x; p < nk; p += blockDim.x) orders[off + p] = sq.ids[best[p]];
  }
  if (threadIdx.x == 0) {
    if (keys) {
      keys[3 * k] = nk > 0 ? h->best_n : -1;
      keys[3 * k + 1] = nk > 0 ? h->best_t : -1;
      keys[3 * k + 2] = nk > 0 ? h->best_chain : -1;
    }
    if (counts) counts[k] = nk;
  }
}

}  // namespace sa
