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
