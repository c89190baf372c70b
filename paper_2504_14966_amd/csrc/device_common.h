// Shared device definitions: the model passed to kernels, the packed request record
// staged in LDS, the workspace layout and 64-lane wavefront helpers.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sa {

constexpr int kWave = 64;

// The kernels one call may run, in order of preference: the first candidate whose needed
// flags the device-side checks of the queue set is the one that runs (the last needs none);
// every other launch returns at once. `allow` are the check flags this launch may use.
struct Gate {
  uint32_t need[4];
  int32_t count;  // candidates (1 .. 4)
  int32_t self;   // this launch's candidate index
  uint32_t allow;
  uint32_t pad;
};

// Integer latency model plus sizes, passed by value to every kernel.
struct DevModel {
  int32_t n;       // requests
  int32_t B;       // max batch
  int32_t policy;  // 0 static, 1 continuous, 2 static with searched batch sizes
  int32_t flags;   // kFlag* widths below (the host's, plus the device checks' allowed by the gate)
  uint64_t p0, p1, d0, d1, d2;
  int64_t t_ref;     // the caller's Metropolis scale (0: total latency of the input order)
  int32_t max_kind;  // largest SLO kind accepted
  int32_t ratio;     // 1: the ratio objective (its cross products must fit int64)
  Gate gate;
};

// One request packed into 16 bytes for a single ds_read_b128 gather:
//   x = l_in | l_out << 16, y = threshold (us), z = kind (low 2 bits), w = prefill cost
//   p0 + p1 * l_in when it fits 32 bits (DevModel flags bit 0).
__device__ __forceinline__ uint32_t req_lin(uint4 r) { return r.x & 0xFFFFu; }
__device__ __forceinline__ uint32_t req_lout(uint4 r) { return r.x >> 16; }

struct QueuePtrs {
  const uint16_t *in_len, *out_len;
  const uint8_t *kind;
  const uint32_t *thr;
};

// 64-bit FNV-1a steps folding the accepted trajectory of a chain.
constexpr uint64_t kFnvOffset = 0xCBF29CE484222325ull;
constexpr uint64_t kFnvPrime = 0x100000001B3ull;

// Workspace layout (bytes), identical on host and device.
struct WsHeader {
  uint64_t magic;
  int32_t n, chains, iters, policy;
  int64_t t_ref, start_n, start_t, allmet;
  int64_t best_chain, best_n, best_t;
  int64_t max_batch;
  int64_t objective, level_len, early_exit;
  // written by the device-side checks of the queue before anything else of a call runs:
  // 0 or a negative SCHED_E* code, the width flags, the candidate kernel that runs (-1: none)
  int64_t plan_status, plan_flags, plan_selected;
  int64_t reserved[13];
};
static_assert(sizeof(WsHeader) <= 256, "header fits its slot");
// Search settings of Algorithm 1: objective 0 = attainment, then total latency; 1 = the
// ratio G = n / t. level_len proposals per temperature level. early_exit: no proposals when
// the solo-latency order meets every SLO.
struct SearchParams {
  int32_t objective, level_len, early_exit, pad;
};

constexpr int kFlagNarrowPrefill = 1;  // continuous event arithmetic fits 32 bits
constexpr int kFlagListSched = 2;      // continuous list scheduling: keys and prefill sums fit
constexpr int kFlagNarrowTime = 4;     // list scheduling: every time on the timeline fits 32 bits
constexpr int kFlagWindows = 8;        // explicit batches: every time below 2^57 (windowed replay)
constexpr int kFlagStaticNarrow = 16;  // static batches of any layout: 24-bit pair costs, 32-bit offsets
constexpr int kFlagTime32 = 32;        // static batches of any layout: every time on the timeline fits 32 bits
constexpr int kFlagFitWindows = 64;    // fitted model: the timeline (and every member's time) below 2^57
constexpr int kFlagFitMember32 = 128;  // fitted model: every member's time, in any batch, below 2^32 - 1
constexpr int kFlagInst64 = 256;       // several instances: each holds at most 64 requests
constexpr int kFlagInst192 = 512;      // several instances: each holds at most 192 requests
constexpr uint64_t kWsMagic = 0x534c4f414e4e3031ull;  // "SLOANN01"

__host__ __device__ __forceinline__ size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }
__host__ __device__ __forceinline__ size_t ws_perm_stride(int n) { return round_up((size_t)n, 128); }  // u16 entries
__host__ __device__ __forceinline__ size_t ws_off_start() { return 256; }
__host__ __device__ __forceinline__ size_t ws_off_records(int n) {
  return ws_off_start() + round_up(2 * (size_t)n, 256);
}
__host__ __device__ __forceinline__ size_t ws_off_cur(int n, int chains) {
  return ws_off_records(n) + round_up((size_t)chains * 64, 256);
}
__host__ __device__ __forceinline__ size_t ws_off_best(int n, int chains) {
  return ws_off_cur(n, chains) + (size_t)chains * ws_perm_stride(n) * 2;
}
// batch layouts of the joint order / batch-size search: one start flag per position
__host__ __device__ __forceinline__ size_t ws_flag_stride(int n) { return round_up((size_t)n, 256); }  // bytes
__host__ __device__ __forceinline__ size_t ws_off_cur_starts(int n, int chains) {
  return ws_off_best(n, chains) + (size_t)chains * ws_perm_stride(n) * 2;
}
__host__ __device__ __forceinline__ size_t ws_off_best_starts(int n, int chains) {
  return ws_off_cur_starts(n, chains) + (size_t)chains * ws_flag_stride(n);
}
__host__ __device__ __forceinline__ size_t ws_total(int n, int chains) {
  return ws_off_best_starts(n, chains) + (size_t)chains * ws_flag_stride(n);
}

// ---- wavefront helpers (64 lanes) ----
__device__ __forceinline__ int lane_id() { return (int)(threadIdx.x & 63u); }

__device__ __forceinline__ void wave_sync_lds() {
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
  __builtin_amdgcn_wave_barrier();
}

__device__ __forceinline__ uint64_t wave_sum_u64(uint64_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}
__device__ __forceinline__ int64_t wave_sum_i64(int64_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}
__device__ __forceinline__ uint32_t wave_min_u32(uint32_t v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = min(v, (uint32_t)__shfl_xor((int)v, o));
  return v;
}
__device__ __forceinline__ int rank_in_mask(uint64_t mask) {
  return (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32), __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}
__device__ __forceinline__ int ballot_count(bool p) { return __popcll(__ballot(p)); }

__device__ __forceinline__ int uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }

}  // namespace sa
