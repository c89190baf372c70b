// Timeline replay of one priority order by one 64-lane wavefront.
//
// Both functions return the objective of the Problem Formulation as the exact integer
// pair (n = requests meeting their SLO, t = sum of end-to-end latencies) and reach the
// value of the one-iteration-at-a-time simulation through closed forms:
//
// Static admission (batch index = position / B; a batch waits for the previous one):
//   all members of a batch start decoding together after one prefill iteration of
//   P = sum(p0 + p1 * l_j). Member m, with L_m output tokens, shares mu_j = min(L_j, L_m)
//   of its decode iterations with member j, and in the s-th of them j holds l_j + s
//   context tokens. Summing the per-token decode model over m's iterations gives
//     F_m = P + L_m * d0 + sum_j [ d1 * mu_j + d2 * (l_j * mu_j + mu_j (mu_j + 1) / 2) ],
//   its finish offset within the batch. The batch lasts max_m F_m, and its start is the
//   sum of the earlier batches' durations (waiting-time equation). Lanes map to batch
//   members: a batch occupies Bp = next power of two >= B lanes and 64 / Bp batches are
//   scored per pass; the start offsets come from a wave prefix sum over the batch leads.
//
// Continuous admission (a finished request frees its slot at the next iteration):
//   lanes are the B slots. Between two events (admission or finish) the running set is
//   fixed, so s decode iterations starting after global decode step K cost
//     s * (d0 + d1 * b + d2 * C) + d2 * b * s (s + 1) / 2,  C = sum over running of
//   (l_in - K0) + b * K (K0 = decode step count at its admission). The loop jumps from
//   event to event with a wave minimum over the slots' finish steps.
#pragma once
#include "device_common.h"

namespace sa {

// Position -> request id of a candidate order, without materialising it.
// kind 0: identity, 1: swap(i, j), 2: insert (remove at i, re-insert at j).
struct Remap {
  int kind, i, j;
  __device__ __forceinline__ int src(int p) const {
    if (kind == 1) return p == i ? j : (p == j ? i : p);
    if (kind == 2) {
      if (i < j) return (p >= i && p < j) ? p + 1 : (p == j ? i : p);
      return p == j ? i : ((p > j && p <= i) ? p - 1 : p);
    }
    return p;
  }
};

struct Score {
  int64_t n;
  uint64_t t;
};

// Apply a move (1 swap, 2 insert: remove at i, re-insert at j) to an order in LDS, in place,
// by one wave. Inserts shift the positions between i and j in chunks of 64, each chunk
// read completely before it is written.
template <typename T>
__device__ __forceinline__ void apply_move_lds(T *perm, int type, int i, int j, int lane) {
  if (type == 1) {
    if (lane == 0) {
      const T x = perm[i];
      perm[i] = perm[j];
      perm[j] = x;
    }
  } else if (type == 2) {
    // shift the positions between i and j by one towards i, 4 x 64 positions per round:
    // the reads of a round cover positions the round's writes do not reach, so one wait
    // per round suffices (LDS accesses of a wave execute in order)
    const T x = perm[i];
    // four named values rather than an array: an array of 16-byte records is not kept in
    // registers by the compiler, which then stages it in scratch memory. A lane past the
    // range writes to position j instead of skipping its store (no branch): j is written
    // last, with the moved entry, and no read of j follows a write to it (reads of a round
    // come first, and only the last round reaches j).
    if (i < j) {
      for (int c0 = i; c0 < j; c0 += 4 * kWave) {
        const int p = c0 + lane;
        const T v0 = perm[min(p + 1, j)], v1 = perm[min(p + kWave + 1, j)];
        const T v2 = perm[min(p + 2 * kWave + 1, j)], v3 = perm[min(p + 3 * kWave + 1, j)];
        perm[min(p, j)] = v0;
        perm[min(p + kWave, j)] = v1;
        perm[min(p + 2 * kWave, j)] = v2;
        perm[min(p + 3 * kWave, j)] = v3;
      }
    } else {
      for (int c0 = i; c0 > j; c0 -= 4 * kWave) {
        const int p = c0 - lane;
        const T v0 = perm[max(p - 1, j)], v1 = perm[max(p - kWave - 1, j)];
        const T v2 = perm[max(p - 2 * kWave - 1, j)], v3 = perm[max(p - 3 * kWave - 1, j)];
        perm[max(p, j)] = v0;
        perm[max(p - kWave, j)] = v1;
        perm[max(p - 2 * kWave, j)] = v2;
        perm[max(p - 3 * kWave, j)] = v3;
      }
    }
    if (lane == 0) perm[j] = x;
  }
  wave_sync_lds();
}

__device__ __forceinline__ bool slo_met(uint32_t kind, uint32_t thr, uint32_t L, uint64_t ttft, uint64_t e2e) {
  if (kind == 0) return ttft <= (uint64_t)thr;
  if (kind == 2) return e2e <= (uint64_t)thr;
  return e2e - ttft <= (uint64_t)thr * (uint64_t)L;
}

// stage: 64-entry per-wave LDS scratch. detail (nullable): 2 int64 per request id.
template <bool DETAIL>
__device__ Score replay_static(const DevModel &m, const uint4 *__restrict__ req, const uint16_t *perm, Remap rm,
                               uint4 *stage, int64_t *detail) {
  const int lane = lane_id();
  const int N = m.n, B = m.B;
  const int lgBp = 32 - __clz(B - 1);  // log2 of the next power of two >= B (B = 1 -> 0)
  const int Bp = 1 << lgBp;
  const int G = kWave >> lgBp;
  const int seg = lane >> lgBp, mm = lane & (Bp - 1);
  const int M = (N + B - 1) / B;
  uint64_t carry = 0, tl = 0;
  int64_t nmet = 0;
  for (int kb = 0; kb < M; kb += G) {
    const int k = kb + seg;
    const int q = k * B + mm;
    const bool valid = (k < M) && (mm < B) && (q < N);
    uint32_t lin = 0, L = 0, thr = 0, kind = 0;
    int r = 0;
    if (valid) {
      r = perm[rm.src(q)];
      const uint4 rq = req[r];
      lin = req_lin(rq);
      L = req_lout(rq);
      thr = rq.y;
      kind = rq.z;
    }
    const uint64_t pf = valid ? m.p0 + m.p1 * (uint64_t)lin : 0;
    stage[lane] = make_uint4(L, lin, (uint32_t)pf, (uint32_t)(pf >> 32));
    wave_sync_lds();
    uint64_t P = 0, acc = 0;
    const int base = seg << lgBp;
    for (int j = 0; j < B; ++j) {
      const uint4 s = stage[base + j];
      P += (uint64_t)s.z | ((uint64_t)s.w << 32);
      const uint64_t mu = min(s.x, L);
      acc += m.d1 * mu + m.d2 * ((uint64_t)s.y * mu + (mu * (mu + 1) >> 1));
    }
    wave_sync_lds();
    const uint64_t F = P + (uint64_t)L * m.d0 + acc;
    uint64_t D = valid ? F : 0;
    for (int o = 1; o < Bp; o <<= 1) D = max(D, (uint64_t)__shfl_xor(D, o));
    uint64_t pre = (mm == 0) ? D : 0;
    for (int o = 1; o < kWave; o <<= 1) {
      const uint64_t y = __shfl_up(pre, o);
      if (lane >= o) pre += y;
    }
    const uint64_t S = carry + pre - D;
    const uint64_t total = __shfl(pre, kWave - 1);
    if (valid) {
      const uint64_t e2e = S + F, ttft = S + P;
      tl += e2e;
      if (DETAIL) {
        detail[2 * r] = (int64_t)ttft;
        detail[2 * r + 1] = (int64_t)e2e;
      }
    }
    bool met = false;
    if (valid) met = slo_met(kind, thr, L, S + P, S + F);
    nmet += ballot_count(met);
    carry += total;
  }
  return Score{nmet, wave_sum_u64(tl)};
}

template <bool DETAIL>
__device__ Score replay_continuous(const DevModel &m, const uint4 *__restrict__ req, const uint16_t *perm, Remap rm,
                                   int64_t *detail) {
  const int lane = lane_id();
  const int N = m.n, B = m.B;
  bool active = false;
  uint32_t fK = 0, L = 0, thr = 0, kind = 0;
  uint64_t ttft = 0;
  int64_t base_r = 0;
  int r = 0;
  uint32_t K = 0;
  uint64_t clock = 0, tl = 0;
  int next = 0, b = 0;
  int64_t base_sum = 0, nmet = 0;
  // every event retires at least one running request, so n events always suffice; the
  // bound only guarantees the loop ends
  for (int ev = 0; ev <= N; ++ev) {
    if (next < N && b < B) {
      const bool is_free = lane < B && !active;
      const int rank = rank_in_mask(__ballot(is_free));
      const int g = min(B - b, N - next);
      const bool adm = is_free && rank < g;
      uint64_t pf = 0;
      if (adm) {
        r = perm[rm.src(next + rank)];
        const uint4 rq = req[r];
        const uint32_t lin = req_lin(rq);
        L = req_lout(rq);
        thr = rq.y;
        kind = rq.z;
        pf = m.p0 + m.p1 * (uint64_t)lin;
        active = true;
        fK = K + L;
        base_r = (int64_t)lin - (int64_t)K;
      }
      clock += wave_sum_u64(pf);
      if (adm) ttft = clock;
      base_sum += wave_sum_i64(adm ? base_r : 0);
      b += g;
      next += g;
    }
    const uint32_t fmin = wave_min_u32(active ? fK : 0xFFFFFFFFu);
    const uint64_t s = (uint64_t)(fmin - K);
    const uint64_t ub = (uint64_t)b;
    const uint64_t C = (uint64_t)(base_sum + (int64_t)ub * (int64_t)K);
    clock += s * (m.d0 + m.d1 * ub + m.d2 * C) + m.d2 * ub * (s * (s + 1) >> 1);
    K = fmin;
    const bool fin = active && fK == K;
    bool met = false;
    if (fin) {
      met = slo_met(kind, thr, L, ttft, clock);
      tl += clock;
      if (DETAIL) {
        detail[2 * r] = (int64_t)ttft;
        detail[2 * r + 1] = (int64_t)clock;
      }
    }
    nmet += ballot_count(met);
    base_sum -= wave_sum_i64(fin ? base_r : 0);
    b -= ballot_count(fin);
    if (fin) active = false;
    if (b == 0 && next >= N) break;
  }
  return Score{nmet, wave_sum_u64(tl)};
}

template <bool DETAIL>
__device__ __forceinline__ Score replay(const DevModel &m, const uint4 *req, const uint16_t *perm, Remap rm,
                                        uint4 *stage, int64_t *detail) {
  if (m.policy != 1) return replay_static<DETAIL>(m, req, perm, rm, stage, detail);  // both static policies
  return replay_continuous<DETAIL>(m, req, perm, rm, detail);
}

}  // namespace sa
