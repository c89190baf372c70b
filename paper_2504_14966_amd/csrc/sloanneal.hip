// C-ABI of the annealing library (declared in include/sloanneal.h): argument checks, workspace
// sizing and kernel launches on the caller's stream. Nothing blocks: the queue's contents are
// checked on the device by each call's first kernel (entries, the int64 range, the integer
// widths that pick the kernel), and every candidate kernel of a call is enqueued behind it,
// of which only the selected one runs.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <functional>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/sloanneal.h"
#include "kernels.h"
#include "anneal_static.h"
#include "anneal_wave.h"
#include "anneal_sized.h"
#include "anneal_wave_rows.h"
#include "anneal_cont_spec.h"
#include "multi.h"
#include "anneal_reg.h"
#include "fit.h"

namespace {

thread_local std::string g_hip_msg;

int hip_fail(hipError_t e) {
  g_hip_msg = hipGetErrorString(e);
  return SCHED_EHIP;
}

#define HIP_TRY(expr)                       \
  do {                                      \
    hipError_t _e = (expr);                 \
    if (_e != hipSuccess) return hip_fail(_e); \
  } while (0)

int check_model(const sched_model_t *m, int n) {
  if (!m) return SCHED_EINVAL;
  if (m->max_batch < 1 || m->max_batch > SCHED_MAX_BATCH) return SCHED_EINVAL;
  if (m->policy != SCHED_STATIC && m->policy != SCHED_CONTINUOUS && m->policy != SCHED_STATIC_SEARCH) return SCHED_EINVAL;
  if (m->p0 < 0 || m->p1 < 0 || m->d0 < 0 || m->d1 < 0 || m->d2 < 0 || m->t_ref_us < 0) return SCHED_EINVAL;
  if (m->swap_threshold > (1ull << 32)) return SCHED_EINVAL;
  (void)n;
  return SCHED_OK;
}

int check_search(const sched_search_t *search, sa::SearchParams &srch) {
  srch = sa::SearchParams{SCHED_OBJ_LEX, 1, 0, 0};
  if (!search) return SCHED_OK;
  if ((search->objective != SCHED_OBJ_LEX && search->objective != SCHED_OBJ_RATIO) || search->level_len < 1 ||
      (search->early_exit != 0 && search->early_exit != 1) || search->reserved != 0)
    return SCHED_EINVAL;
  srch = sa::SearchParams{search->objective, search->level_len, search->early_exit, 0};
  return SCHED_OK;
}
int check_chain_args(int32_t chains, int32_t iters, double T0, double alpha) {
  if (chains < 1 || iters < 0 || !(T0 > 0.0) || !std::isfinite(T0) || !(alpha > 0.0) || !std::isfinite(alpha))
    return SCHED_EINVAL;
  return SCHED_OK;
}

// Host-side checks of a queue descriptor (its contents are checked on the device).
int check_queue(const sched_queue_t *q) {
  if (!q || q->n < 1 || q->n > SCHED_MAX_N) return SCHED_EINVAL;
  if (!q->in_len || !q->out_len || !q->kind || !q->thr_us) return SCHED_EINVAL;
  return SCHED_OK;
}

// The fitted model: every coefficient >= 0, batches of 1 .. 64.
int check_fit(const sched_fit_model_t *f) {
  if (!f || f->max_batch < 1 || f->max_batch > SCHED_MAX_BATCH) return SCHED_EINVAL;
  if (f->policy != SCHED_STATIC && f->policy != SCHED_STATIC_SEARCH) return SCHED_EINVAL;
  if (f->ap < 0 || f->bp < 0 || f->cp < 0 || f->dp < 0 || f->ad < 0 || f->bd < 0 || f->cd < 0 || f->dd < 0 ||
      f->t_ref < 0 || f->swap_threshold > (1ull << 32))
    return SCHED_EINVAL;
  return SCHED_OK;
}

// Width flags each kernel may take from the device checks (the device adds the ones that
// hold for the queue): single-queue annealing, evaluation and several instances.
constexpr uint32_t kAnnealFlags = sa::kFlagNarrowPrefill | sa::kFlagListSched | sa::kFlagNarrowTime | sa::kFlagWindows;
constexpr uint32_t kEvalFlags = sa::kFlagNarrowPrefill | sa::kFlagListSched | sa::kFlagNarrowTime;
constexpr uint32_t kMultiFlags = kEvalFlags;
constexpr uint32_t kSN = sa::kFlagStaticNarrow, kT32 = sa::kFlagTime32;

// The kernels one call may run, in order of preference, each with the width flags it needs
// and the ones it may use. All of them are enqueued; on the device each reads the verdict of
// the checks and only the first whose needs hold runs (the last needs none, so exactly one
// runs when the queue passes the checks, none when it fails them).
template <class M>
struct Candidates {
  sa::Gate gate{};
  uint32_t allow[4] = {0u, 0u, 0u, 0u};
  std::function<hipError_t(const M &)> launch[4];
  void add(uint32_t need, uint32_t allow_flags, std::function<hipError_t(const M &)> fn) {
    if (gate.count >= 4) return;  // at most three per call by construction
    gate.need[gate.count] = need;
    allow[gate.count] = allow_flags;
    launch[gate.count] = std::move(fn);
    ++gate.count;
  }
  // The model of the kernel that runs the checks: every candidate's needs, its own flags.
  M checker(M m, uint32_t allow_flags) const {
    m.gate = gate;
    m.gate.self = -1;
    m.gate.allow = allow_flags;
    return m;
  }
  int run(const M &m) const {
    if (gate.count < 1 || gate.need[gate.count - 1] != 0u) return SCHED_EINVAL;
    for (int c = 0; c < gate.count; ++c) {
      M mc = checker(m, allow[c]);
      mc.gate.self = c;
      const hipError_t e = launch[c](mc);
      if (e != hipSuccess) return hip_fail(e);
    }
    return SCHED_OK;
  }
};

// max_kind: the largest SLO kind the call accepts; ratio: the ratio objective.
sa::DevModel dev_model(const sched_model_t *m, int n, int max_kind = 2, int ratio = 0) {
  sa::DevModel d{};
  d.n = n;
  d.B = m->max_batch;
  d.policy = m->policy;
  d.flags = 0;
  d.p0 = (uint64_t)m->p0;
  d.p1 = (uint64_t)m->p1;
  d.d0 = (uint64_t)m->d0;
  d.d1 = (uint64_t)m->d1;
  d.d2 = (uint64_t)m->d2;
  d.t_ref = m->t_ref_us;
  d.max_kind = max_kind;
  d.ratio = ratio;
  return d;
}

sa::DevFit dev_fit(const sched_fit_model_t *f, int n, int max_kind, int ratio) {
  sa::DevFit d{};
  d.n = n;
  d.B = f->max_batch;
  d.policy = f->policy;
  d.ap = (uint64_t)f->ap;
  d.bp = (uint64_t)f->bp;
  d.cp = (uint64_t)f->cp;
  d.dp = (uint64_t)f->dp;
  d.ad = (uint64_t)f->ad;
  d.bd = (uint64_t)f->bd;
  d.cd = (uint64_t)f->cd;
  d.dd = (uint64_t)f->dd;
  d.win = 0u;
  d.m32 = 0u;
  d.bmagic = (1ull << 32) / (uint64_t)f->max_batch + 1;
  d.t_ref = f->t_ref;
  d.max_kind = max_kind;
  d.ratio = ratio;
  return d;
}

sa::QueuePtrs dev_queue(const sched_queue_t *q) {
  return sa::QueuePtrs{q->in_len, q->out_len, q->kind, q->thr_us};
}

size_t eval_lds_bytes(int n, bool ls, int waves) {
  const size_t per_wave = ((size_t)n * 2 + 15) / 16 * 16 + 64 * 16 + 32 * 4 +
                          (ls ? (sa::cont_ls_scratch_bytes(n) + 15) / 16 * 16 : 0);
  return ((size_t)n * 16 + 15) / 16 * 16 + per_wave * waves;
}

size_t static_wave_lds(int n, int B) { return sa::static_chain_bytes(n, B); }
size_t wave_chain_lds(int n, int B) { return sa::wave_chain_bytes(n, B); }

int device_attr(hipDeviceAttribute_t attr, int fallback) {
  int dev = 0, v = 0;
  if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&v, attr, dev) != hipSuccess) return fallback;
  return v;
}
int max_lds_per_block() { return device_attr(hipDeviceAttributeMaxSharedMemoryPerBlock, 65536); }
int cu_count() { return device_attr(hipDeviceAttributeMultiprocessorCount, 256); }

size_t sized_chain_lds(int n) {
  const size_t pb = ((size_t)n * 2 + 15) & ~size_t(15), fb = ((size_t)n + 15) & ~size_t(15);
  const size_t ub = ((size_t)n * 4 + 15) & ~size_t(15);
  return pb + fb + ub;
}

size_t anneal_lds_bytes(int n) {
  const size_t per_wave = ((size_t)n * 2 + 15) / 16 * 16 * 2 + 64 * 16;
  return ((size_t)n * 16 + 15) / 16 * 16 + per_wave * sa::kWavesPerBlock;
}

// Chains per workgroup of the register kernels: four, or fewer so that the chains spread
// over every CU.
int reg_waves(int chains) {
  const int cus = std::max(1, cu_count());
  return chains >= 4 * cus ? 4 : (chains >= 2 * cus ? 2 : 1);
}

// Everything one sched_anneal launch needs besides the model and the gate.
struct ChainArgs {
  sa::QueuePtrs q;
  int chains, iters;
  double T0, alpha;
  uint32_t k0, k1;
  uint64_t swap_thr;
  sa::SearchParams srch;
  unsigned char *w;
  hipStream_t stream;
};

static_assert(sa::sized_rows_for(SCHED_MAX_N) * 64 >= SCHED_MAX_N, "register rows must cover every position");
static_assert(sa::limit_rows_for((SCHED_MAX_N + 32) / 33) * 33 >= SCHED_MAX_N,
              "limit rows must cover every batch when batches hold 33 or more");

template <int OBJ, int NR>
hipError_t launch_sized(int grid, int waves, size_t lds, const sa::DevModel &d, const sa::StaticParams &sp,
                        const ChainArgs &a) {
  if (lds > 65536) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(&sa::anneal_sized_kernel<OBJ, NR>),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  sa::anneal_sized_kernel<OBJ, NR><<<grid, waves * 64, lds, a.stream>>>(d, sp, a.q, a.chains, a.iters, a.T0, a.alpha,
                                                                        a.k0, a.k1, a.srch, a.w);
  return hipGetLastError();
}

// The joint order / batch-size search: on small queues the register kernel (order, request
// fields and layout in registers, no LDS) when the 32-bit pair-cost widths hold; else the
// delta kernel when the widths and the whole timeline fit 32 bits (as many chains per
// workgroup as spread the chains over every CU, at most 16 and at most what the LDS holds);
// the full-replay kernel, four chains per workgroup, in any case.
template <int OBJ>
void add_sized(Candidates<sa::DevModel> &c, const sched_model_t *model, int n, const ChainArgs &a) {
  if (sa::reg_sized_fits(n)) {
    const int waves = reg_waves(a.chains), grid = (a.chains + waves - 1) / waves;
    c.add(kSN, kAnnealFlags | kT32, [=](const sa::DevModel &d) {
      sa::anneal_reg_sized_kernel<OBJ><<<grid, waves * 64, 0, a.stream>>>(d, a.q, a.chains, a.iters, a.T0, a.alpha,
                                                                         a.k0, a.k1, a.srch, a.w);
      return hipGetLastError();
    });
  } else {
    const size_t soa = (size_t)(n + 1) * 16, per = sized_chain_lds(n);
    const int lim = max_lds_per_block(), cus = std::max(1, cu_count());
    int waves = 1;
    while (waves < 16 && (int64_t)waves * cus < a.chains) waves <<= 1;
    while (waves > 1 && soa + per * waves > (size_t)lim) waves >>= 1;
    if (soa + per * waves <= (size_t)lim) {
      const size_t lds = soa + per * waves;
      const sa::StaticParams sp{(uint32_t)model->d0, (uint32_t)model->d2, (1ull << 32) / (uint64_t)model->max_batch + 1};
      const int grid = (a.chains + waves - 1) / waves;
      const int rows = sa::sized_rows_for(n);
      c.add(kSN | kT32, kAnnealFlags, [=](const sa::DevModel &d) {
        switch (rows) {
          case 2: return launch_sized<OBJ, 2>(grid, waves, lds, d, sp, a);
          case 4: return launch_sized<OBJ, 4>(grid, waves, lds, d, sp, a);
          case 8: return launch_sized<OBJ, 8>(grid, waves, lds, d, sp, a);
          default: return launch_sized<OBJ, 16>(grid, waves, lds, d, sp, a);
        }
      });
    }
  }
  const size_t pb = ((size_t)n * 2 + 15) & ~size_t(15), fb = ((size_t)n + 15) & ~size_t(15);
  const size_t lds = (((size_t)n * 16 + 15) & ~size_t(15)) + 4 * (2 * pb + 2 * fb + 64 * 16);
  const int grid = (a.chains + 3) / 4;
  c.add(0u, kAnnealFlags, [=](const sa::DevModel &d) {
    sa::anneal_sized_generic_kernel<OBJ><<<grid, 256, lds, a.stream>>>(d, a.q, a.chains, a.iters, a.T0, a.alpha, a.k0,
                                                                       a.k1, a.srch, a.w);
    return hipGetLastError();
  });
}

template <int LG, int OBJ>
hipError_t launch_reg(bool parts, int grid, int waves, const sa::DevModel &d, const ChainArgs &a) {
  if (parts)
    sa::anneal_reg_h_kernel<LG, OBJ><<<grid, waves * 64, 0, a.stream>>>(d, a.q, a.chains, a.iters, a.T0, a.alpha, a.k0,
                                                                        a.k1, a.swap_thr, a.srch, a.w);
  else
    sa::anneal_reg_kernel<LG, OBJ><<<grid, waves * 64, 0, a.stream>>>(d, a.q, a.chains, a.iters, a.T0, a.alpha, a.k0,
                                                                      a.k1, a.swap_thr, a.srch, a.w);
  return hipGetLastError();
}

template <int OBJ, int MR>
hipError_t launch_rows(int waves, size_t lds, const sa::DevModel &d, const sa::StaticParams &sp, const ChainArgs &a) {
  if (lds > 65536) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(&sa::anneal_rows_kernel<OBJ, MR>),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  const int grid = (a.chains + waves - 1) / waves;
  sa::anneal_rows_kernel<OBJ, MR><<<grid, waves * 64, lds, a.stream>>>(d, sp, a.q, a.chains, a.iters, a.T0, a.alpha,
                                                                       a.k0, a.k1, a.swap_thr, a.srch, a.w);
  return hipGetLastError();
}

template <int LG, int OBJ>
hipError_t launch_static(int waves, size_t lds, const sa::DevModel &d, const sa::StaticParams &sp, const ChainArgs &a) {
  const void *fn = LG == 6 ? reinterpret_cast<const void *>(&sa::anneal_wave_kernel<OBJ>)
                           : reinterpret_cast<const void *>(&sa::anneal_static_kernel<LG, OBJ>);
  if (lds > 65536) {
    const hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  const int grid = (a.chains + waves - 1) / waves;
  if constexpr (LG == 6)
    sa::anneal_wave_kernel<OBJ><<<grid, waves * 64, lds, a.stream>>>(d, sp, a.q, a.chains, a.iters, a.T0, a.alpha, a.k0,
                                                                     a.k1, a.swap_thr, a.srch, a.w);
  else
    sa::anneal_static_kernel<LG, OBJ><<<grid, waves * 64, lds, a.stream>>>(d, sp, a.q, a.chains, a.iters, a.T0,
                                                                           a.alpha, a.k0, a.k1, a.swap_thr, a.srch,
                                                                           a.w);
  return hipGetLastError();
}

// The kernels a single-queue sched_anneal may run, by policy, in order of preference:
//   static: the register kernel (up to 64 requests, or 65 to 192 with two or three positions
//     per lane; batches of 1 .. 16, a power of two) or else the LDS delta kernel (one lane per
//     batch member, or one batch per wave for batches of more than 32), both on the 32-bit
//     pair-cost widths, the register kernel also on a 32-bit timeline when it holds, and
//     one batch per wave with the members' SLO limits in registers ahead of the plain one
//     when the timeline fits 32 bits;
//   continuous: list scheduling when its 32-bit keys fit, the event loop when the 32-bit event
//     arithmetic does, each as the LDS allows;
//   always last: the full-replay kernel (any widths).
template <int OBJ>
void add_chains(Candidates<sa::DevModel> &c, const sched_model_t *model, int n, const ChainArgs &a) {
  const int B = model->max_batch;
  if (model->policy == SCHED_STATIC_SEARCH) {
    add_sized<OBJ>(c, model, n, a);
    return;
  }
  if (model->policy == SCHED_STATIC) {
    if (sa::reg_kernel_fits(n, B) || sa::reg_parts(n, B) > 1) {
      const bool parts = !sa::reg_kernel_fits(n, B);
      const int waves = reg_waves(a.chains), grid = (a.chains + waves - 1) / waves;
      c.add(kSN, kAnnealFlags | kT32, [=](const sa::DevModel &d) {
        switch (B) {
          case 1: return launch_reg<0, OBJ>(parts, grid, waves, d, a);
          case 2: return launch_reg<1, OBJ>(parts, grid, waves, d, a);
          case 4: return launch_reg<2, OBJ>(parts, grid, waves, d, a);
          case 8: return launch_reg<3, OBJ>(parts, grid, waves, d, a);
          default: return launch_reg<4, OBJ>(parts, grid, waves, d, a);
        }
      });
    } else {
      // chains per workgroup: enough to spread the chains over every CU, at most 16 and at
      // most what the LDS holds
      int lg = 0;
      while ((1 << lg) < B) ++lg;
      const size_t soa = (size_t)(n + 1) * 16;
      const size_t per = lg == 6 ? wave_chain_lds(n, B) : static_wave_lds(n, B);
      const int lim = max_lds_per_block(), cus = std::max(1, cu_count());
      int waves = 1;
      while (waves < 16 && (int64_t)waves * cus < a.chains) waves <<= 1;
      while (waves > 1 && soa + per * waves > (size_t)lim) waves >>= 1;
      if (soa + per * waves <= (size_t)lim && (waves >= 4 || (int64_t)waves * cus >= a.chains)) {
        const sa::StaticParams sp{(uint32_t)model->d0, (uint32_t)model->d2, (1ull << 32) / (uint64_t)B + 1};
        const size_t lds = soa + per * waves;
        if (lg == 6) {
          // the limit-row kernel when the whole timeline fits 32 bits (its chains take a
          // little more LDS: the order carries 64 spare entries)
          const size_t rper = sa::rows_chain_bytes(n, B);
          int rwaves = waves;
          while (rwaves > 1 && soa + rper * rwaves > (size_t)lim) rwaves >>= 1;
          const size_t rlds = soa + rper * rwaves;
          const int rows = sa::limit_rows_for((n + B - 1) / B);
          if (rlds <= (size_t)lim && (rwaves >= 4 || (int64_t)rwaves * cus >= a.chains))
            c.add(kSN | kT32, kAnnealFlags, [=](const sa::DevModel &d) {
              switch (rows) {
                case 8: return launch_rows<OBJ, 8>(rwaves, rlds, d, sp, a);
                case 16: return launch_rows<OBJ, 16>(rwaves, rlds, d, sp, a);
                default: return launch_rows<OBJ, 32>(rwaves, rlds, d, sp, a);
              }
            });
        }
        c.add(kSN, kAnnealFlags, [=](const sa::DevModel &d) {
          switch (lg) {
            case 0: return launch_static<0, OBJ>(waves, lds, d, sp, a);
            case 1: return launch_static<1, OBJ>(waves, lds, d, sp, a);
            case 2: return launch_static<2, OBJ>(waves, lds, d, sp, a);
            case 3: return launch_static<3, OBJ>(waves, lds, d, sp, a);
            case 4: return launch_static<4, OBJ>(waves, lds, d, sp, a);
            case 5: return launch_static<5, OBJ>(waves, lds, d, sp, a);
            default: return launch_static<6, OBJ>(waves, lds, d, sp, a);
          }
        });
      }
    }
  }
  if (model->policy == SCHED_CONTINUOUS) {
    // Two proposals scored per round by two waves of one workgroup per chain (list
    // scheduling, 32-bit times), when at least as many chains fit on a CU at once as under
    // the single-proposal list-scheduling kernel.
    {
      const int cus = std::max(1, cu_count()), lim = max_lds_per_block();
      int w1 = 1;
      while (w1 < 16 && (int64_t)w1 * cus < a.chains) w1 <<= 1;
      const size_t per1 = (((size_t)n * 2 + 15) & ~size_t(15)) + ((sa::cont_ls_scratch_bytes(n) + 15) & ~size_t(15)) +
                          (std::min(B, n) <= 32 ? sa::cont_inc_bytes(n, B) : 0);
      while (w1 > 1 && (size_t)n * 16 + per1 * w1 > (size_t)lim) w1 >>= 1;
      const size_t lds1 = (size_t)n * 16 + per1 * w1;
      const int64_t res1 = lds1 <= (size_t)lim ? (int64_t)w1 * std::max<int64_t>(1, lim / (int64_t)lds1) : 0;
      const size_t lds = sa::spec_chain_bytes(n, B);
      const void *fn = (const void *)&sa::anneal_cont_spec_kernel<OBJ>;
      int nb = 0;
      if (lds > (size_t)lim ||
          (lds > 65536 && hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds) != hipSuccess) ||
          hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, fn, 128, lds) != hipSuccess)
        nb = 0;
      if (nb > 0 && std::min<int64_t>(a.chains, (int64_t)nb * cus) >= std::min<int64_t>(a.chains, res1 * cus)) {
        c.add(sa::kFlagNarrowPrefill | sa::kFlagListSched | sa::kFlagNarrowTime, kAnnealFlags,
              [=](const sa::DevModel &d) {
                sa::anneal_cont_spec_kernel<OBJ><<<a.chains, 128, lds, a.stream>>>(
                    d, a.q, a.chains, a.iters, a.T0, a.alpha, a.k0, a.k1, a.swap_thr, a.srch, a.w);
                return hipGetLastError();
              });
      }
    }
    for (int ls = 1; ls >= 0; --ls) {
      const size_t soa = (size_t)n * 16;
      const bool inc = ls && std::min(B, n) <= 32;
      const size_t per = (((size_t)n * 2 + 15) & ~size_t(15)) +
                         (ls ? ((sa::cont_ls_scratch_bytes(n) + 15) & ~size_t(15)) : 0) +
                         (inc ? sa::cont_inc_bytes(n, B) : 0);
      const int cus = std::max(1, cu_count()), lim = max_lds_per_block();
      int waves = 1;
      while (waves < 16 && (int64_t)waves * cus < a.chains) waves <<= 1;
      while (waves > 1 && soa + per * waves > (size_t)lim) waves >>= 1;
      const size_t lds = soa + per * waves;
      if (lds > (size_t)lim) continue;
      const int grid = (a.chains + waves - 1) / waves;
      const uint32_t need = sa::kFlagNarrowPrefill | (ls ? sa::kFlagListSched : 0u);
      c.add(need, kAnnealFlags, [=](const sa::DevModel &d) {
        const void *fn = ls ? (const void *)&sa::anneal_cont_kernel<true, OBJ>
                            : (const void *)&sa::anneal_cont_kernel<false, OBJ>;
        if (lds > 65536) {
          const hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
          if (e != hipSuccess) return e;
        }
        if (ls)
          sa::anneal_cont_kernel<true, OBJ><<<grid, waves * 64, lds, a.stream>>>(d, a.q, a.chains, a.iters, a.T0, a.alpha,
                                                                                 a.k0, a.k1, a.swap_thr, a.srch, a.w);
        else
          sa::anneal_cont_kernel<false, OBJ><<<grid, waves * 64, lds, a.stream>>>(
              d, a.q, a.chains, a.iters, a.T0, a.alpha, a.k0, a.k1, a.swap_thr, a.srch, a.w);
        return hipGetLastError();
      });
    }
  }
  const int grid = (a.chains + sa::kWavesPerBlock - 1) / sa::kWavesPerBlock;
  const size_t lds = anneal_lds_bytes(n);
  c.add(0u, kAnnealFlags, [=](const sa::DevModel &d) {
    sa::anneal_kernel<OBJ><<<grid, sa::kBlock, lds, a.stream>>>(d, a.q, a.chains, a.iters, a.T0, a.alpha, a.k0, a.k1,
                                                                a.swap_thr, a.srch, a.w);
    return hipGetLastError();
  });
}

// Everything one sched_anneal_multi launch needs besides the model and the gate.
struct MultiArgs {
  int n, instances, chains, iters;
  double T0, alpha;
  uint32_t k0, k1;
  uint64_t swap_thr;
  sa::SearchParams srch;
  unsigned char *w;
  hipStream_t stream;
};

template <int LG, int OBJ>
hipError_t launch_multi_reg(bool parts, int grid, int waves, int groups, const sa::DevModel &d, const MultiArgs &a) {
  if (parts)
    sa::multi_reg_h_kernel<LG, OBJ><<<grid, waves * 64, 0, a.stream>>>(d, a.n, a.instances, a.chains, groups, a.iters,
                                                                       a.T0, a.alpha, a.k0, a.k1, a.swap_thr, a.srch,
                                                                       a.w);
  else
    sa::multi_reg_kernel<LG, OBJ><<<grid, waves * 64, 0, a.stream>>>(d, a.n, a.instances, a.chains, groups, a.iters,
                                                                     a.T0, a.alpha, a.k0, a.k1, a.swap_thr, a.srch,
                                                                     a.w);
  return hipGetLastError();
}

template <int LG, int OBJ>
hipError_t launch_multi_static(int grid, int waves, int groups, size_t lds, const sa::DevModel &d,
                               const sa::StaticParams &sp, const MultiArgs &a) {
  if (lds > 65536) {
    const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(&sa::multi_static_kernel<LG, OBJ>),
                                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  sa::multi_static_kernel<LG, OBJ><<<grid, waves * 64, lds, a.stream>>>(d, sp, a.n, a.instances, a.chains, groups,
                                                                        a.iters, a.T0, a.alpha, a.k0, a.k1, a.swap_thr,
                                                                        a.srch, a.w);
  return hipGetLastError();
}

// The kernels a sched_anneal_multi may run, in order of preference (static admission):
// the register kernel when every instance holds at most 64 requests, its two- and
// three-position form when every instance holds at most 192 (batches of 1 .. 16, a power of
// two, on the 32-bit pair-cost widths); the LDS delta kernels, laid out for the whole queue
// (an instance never holds more); always last the full-replay kernel (LDS for the whole
// queue too).
template <int OBJ>
void add_multi(Candidates<sa::DevModel> &c, const sched_model_t *model, const MultiArgs &a) {
  const int B = model->max_batch, n = a.n, total = a.instances * a.chains;
  const int cus = std::max(1, cu_count());
  if (model->policy == SCHED_STATIC && sa::reg_parts(1, B) > 0) {
    const int waves = total >= 4 * cus && a.chains >= 4 ? 4 : (total >= 2 * cus && a.chains >= 2 ? 2 : 1);
    const int groups = (a.chains + waves - 1) / waves, grid = a.instances * groups;
    for (int parts = 0; parts <= 1; ++parts) {
      c.add(kSN | (parts ? sa::kFlagInst192 : sa::kFlagInst64), kMultiFlags | kT32, [=](const sa::DevModel &d) {
        switch (B) {
          case 1: return launch_multi_reg<0, OBJ>(parts, grid, waves, groups, d, a);
          case 2: return launch_multi_reg<1, OBJ>(parts, grid, waves, groups, d, a);
          case 4: return launch_multi_reg<2, OBJ>(parts, grid, waves, groups, d, a);
          case 8: return launch_multi_reg<3, OBJ>(parts, grid, waves, groups, d, a);
          default: return launch_multi_reg<4, OBJ>(parts, grid, waves, groups, d, a);
        }
      });
    }
  }
  if (model->policy == SCHED_STATIC) {
    int lg = 0;
    while ((1 << lg) < B) ++lg;
    const size_t soa = (size_t)(n + 1) * 16;
    const size_t per = lg == 6 ? wave_chain_lds(n, B) : static_wave_lds(n, B);
    const int lim = max_lds_per_block();
    int waves = 1;
    while (waves < 16 && waves < a.chains && (int64_t)waves * cus < total) waves <<= 1;
    while (waves > 1 && soa + per * waves > (size_t)lim) waves >>= 1;
    if (soa + per * waves <= (size_t)lim && (waves >= 4 || (int64_t)waves * cus >= total)) {
      const sa::StaticParams sp{(uint32_t)model->d0, (uint32_t)model->d2, (1ull << 32) / (uint64_t)B + 1};
      const size_t lds = soa + per * waves;
      const int groups = (a.chains + waves - 1) / waves, grid = a.instances * groups;
      c.add(kSN, kMultiFlags, [=](const sa::DevModel &d) {
        switch (lg) {
          case 0: return launch_multi_static<0, OBJ>(grid, waves, groups, lds, d, sp, a);
          case 1: return launch_multi_static<1, OBJ>(grid, waves, groups, lds, d, sp, a);
          case 2: return launch_multi_static<2, OBJ>(grid, waves, groups, lds, d, sp, a);
          case 3: return launch_multi_static<3, OBJ>(grid, waves, groups, lds, d, sp, a);
          case 4: return launch_multi_static<4, OBJ>(grid, waves, groups, lds, d, sp, a);
          case 5: return launch_multi_static<5, OBJ>(grid, waves, groups, lds, d, sp, a);
          default: return launch_multi_static<6, OBJ>(grid, waves, groups, lds, d, sp, a);
        }
      });
    }
  }
  const int groups = (a.chains + sa::kWavesPerBlock - 1) / sa::kWavesPerBlock;
  const size_t lds = anneal_lds_bytes(n);
  c.add(0u, kMultiFlags, [=](const sa::DevModel &d) {
    sa::multi_anneal_kernel<OBJ><<<a.instances * groups, sa::kBlock, lds, a.stream>>>(
        d, a.n, a.instances, a.chains, groups, a.iters, a.T0, a.alpha, a.k0, a.k1, a.swap_thr, a.srch, a.w);
    return hipGetLastError();
  });
}

// Fixed device scratch of sched_anneal_noalloc: the annealing workspace for callers that
// cannot allocate. Each GPU the library runs on holds its own copy until the process ends.
// Host code never passes the array's name to a kernel (on the host it is only a stand-in for
// the symbol); it uses the device address obtained once per device below.
static __device__ __align__(256) unsigned char scratch[SCHED_NOALLOC_MAX_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};

// Address of the current device's copy of `scratch`, looked up on the first call on that
// device with the device current.
int scratch_address(void **out) {
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) return SCHED_EINVAL;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void *p = nullptr;
    HIP_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) return SCHED_EHIP;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return SCHED_OK;
}

}  // namespace

extern "C" {

int sched_eval(const sched_queue_t *queue, const sched_model_t *model, const uint16_t *perms, int64_t k, int64_t *out,
               int64_t *detail, hipStream_t stream) {
  if (k < 0) return SCHED_EINVAL;
  int rc = check_queue(queue);
  if (rc) return rc;
  if ((rc = check_model(model, queue->n))) return rc;
  if (k > 0 && (!perms || !out)) return SCHED_EINVAL;
  if (k == 0) return SCHED_OK;
  const int n = queue->n;
  const sa::DevModel dm = dev_model(model, n);
  const sa::QueuePtrs qp = dev_queue(queue);
  Candidates<sa::DevModel> c;
  if (model->policy != SCHED_CONTINUOUS) {
    // static batches on the 32-bit pair-cost widths: one order per wave with the delta
    // kernels' arithmetic, on a 32-bit timeline when it holds
    int lg = 0;
    while ((1 << lg) < model->max_batch) ++lg;
    const sa::StaticParams sp{(uint32_t)model->d0, (uint32_t)model->d2, (1ull << 32) / (uint64_t)model->max_batch + 1};
    const size_t lds = (size_t)(n + 1) * 16 + ((((size_t)n * 2 + 15) & ~size_t(15)) + 64 * 8 + 32 * 4) * 4;
    const int g4 = (int)std::min<int64_t>((k + 3) / 4, 256 * 32);
    auto launch = [=](const sa::DevModel &d, bool t32) {
#define SA_EVAL_CASE(L)                                                                                        \
  case L:                                                                                                      \
    if (detail)                                                                                                \
      sa::eval_static_kernel<L, true><<<g4, 256, lds, stream>>>(d, sp, qp, perms, k, out, detail);             \
    else if (t32)                                                                                              \
      sa::eval_static_kernel<L, false, true><<<g4, 256, lds, stream>>>(d, sp, qp, perms, k, out, nullptr);     \
    else                                                                                                       \
      sa::eval_static_kernel<L, false><<<g4, 256, lds, stream>>>(d, sp, qp, perms, k, out, nullptr);           \
    break;
      switch (lg) {
        SA_EVAL_CASE(0)
        SA_EVAL_CASE(1)
        SA_EVAL_CASE(2)
        SA_EVAL_CASE(3)
        SA_EVAL_CASE(4)
        SA_EVAL_CASE(5)
        default:
          SA_EVAL_CASE(6)
      }
#undef SA_EVAL_CASE
      return hipGetLastError();
    };
    if (!detail) c.add(kSN | kT32, kEvalFlags, [=](const sa::DevModel &d) { return launch(d, true); });
    c.add(kSN, kEvalFlags, [=](const sa::DevModel &d) { return launch(d, false); });
  }
  // any widths: one order per wave, up to four waves per workgroup as the LDS allows (with
  // room for list scheduling under continuous admission)
  const bool ls = model->policy == SCHED_CONTINUOUS;
  const size_t lim = (size_t)max_lds_per_block() - sa::kCheckLdsBytes;  // the checks' own LDS on top
  int waves = sa::kWavesPerBlock;
  while (waves > 1 && eval_lds_bytes(n, ls, waves) > lim) waves >>= 1;
  const size_t lds = eval_lds_bytes(n, ls, waves);
  const int grid = (int)std::min<int64_t>((k + waves - 1) / waves, 256 * 32);
  auto generic = [=](const sa::DevModel &d, int g) {
    const void *fn = detail ? (const void *)&sa::eval_kernel<true> : (const void *)&sa::eval_kernel<false>;
    if (lds > 65536) {
      const hipError_t e = hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
      if (e != hipSuccess) return e;
    }
    if (detail)
      sa::eval_kernel<true><<<g, waves * 64, lds, stream>>>(d, qp, perms, k, out, detail);
    else
      sa::eval_kernel<false><<<g, waves * 64, lds, stream>>>(d, qp, perms, k, out, nullptr);
    return hipGetLastError();
  };
  c.add(0u, kEvalFlags, [=](const sa::DevModel &d) { return generic(d, grid); });
  if ((rc = c.run(dm)) || c.gate.count < 2) return rc;
  // row 0 when a candidate other than the first replayed the rest (its verdict marker sits
  // there until now)
  sa::DevModel fix = c.checker(dm, kEvalFlags);
  fix.gate.self = sa::kEvalFixup;
  const hipError_t e = generic(fix, 1);
  return e == hipSuccess ? SCHED_OK : hip_fail(e);
}

size_t sched_ws_bytes(int32_t n, int32_t chains) {
  if (n < 1 || n > SCHED_MAX_N || chains < 1) return 0;
  return sa::ws_total(n, chains);
}

int sched_anneal(const sched_queue_t *queue, const sched_model_t *model, int32_t chains, int32_t iters, double T0,
                 double alpha, uint64_t seed, void *ws, size_t ws_bytes, hipStream_t stream) {
  return sched_anneal_ex(queue, model, nullptr, chains, iters, T0, alpha, seed, ws, ws_bytes, stream);
}

int sched_anneal_ex(const sched_queue_t *queue, const sched_model_t *model, const sched_search_t *search,
                    int32_t chains, int32_t iters, double T0, double alpha, uint64_t seed, void *ws, size_t ws_bytes,
                    hipStream_t stream) {
  int rc = check_queue(queue);
  if (rc) return rc;
  if ((rc = check_chain_args(chains, iters, T0, alpha))) return rc;
  sa::SearchParams srch;
  if ((rc = check_search(search, srch))) return rc;
  if ((rc = check_model(model, queue->n))) return rc;
  // the ratio needs a positive total latency: every request takes at least p0 + d0 + d1
  if (srch.objective == SCHED_OBJ_RATIO && model->p0 + model->d0 + model->d1 < 1) return SCHED_EINVAL;
  if (!ws || (reinterpret_cast<uintptr_t>(ws) & 255u)) return SCHED_EINVAL;
  if (ws_bytes < sched_ws_bytes(queue->n, chains)) return SCHED_ENOSPC;
  const int n = queue->n;
  const sa::DevModel dm = dev_model(model, n, 2, srch.objective == SCHED_OBJ_RATIO);
  unsigned char *w = static_cast<unsigned char *>(ws);
  const ChainArgs a{dev_queue(queue), chains, iters, T0, alpha, (uint32_t)seed, (uint32_t)(seed >> 32),
                    model->swap_threshold, srch, w, stream};
  Candidates<sa::DevModel> c;
  if (srch.objective)
    add_chains<1>(c, model, n, a);
  else
    add_chains<0>(c, model, n, a);
  sa::start_kernel<<<1, 1024, 0, stream>>>(c.checker(dm, kAnnealFlags), a.q, chains, iters, model->t_ref_us, srch, w);
  HIP_TRY(hipGetLastError());
  if ((rc = c.run(dm))) return rc;
  sa::reduce_kernel<<<1, 1024, 0, stream>>>(w);
  HIP_TRY(hipGetLastError());
  return SCHED_OK;
}

int sched_anneal_noalloc(const sched_queue_t *queue, const sched_model_t *model, int32_t chains, int32_t iters,
                         double T0, double alpha, uint64_t seed, uint16_t *perm_out, int64_t *key_out,
                         hipStream_t stream) {
  if (!queue || queue->n < 1 || queue->n > SCHED_MAX_N || chains < 1) return SCHED_EINVAL;
  if (!perm_out || !key_out) return SCHED_EINVAL;
  if (sched_ws_bytes(queue->n, chains) > (size_t)SCHED_NOALLOC_MAX_BYTES) return SCHED_ENOSPC;
  void *ws = nullptr;
  int rc = scratch_address(&ws);
  if (rc) return rc;
  rc = sched_anneal_ex(queue, model, nullptr, chains, iters, T0, alpha, seed, ws, (size_t)SCHED_NOALLOC_MAX_BYTES,
                       stream);
  if (rc) return rc;
  return sched_best(ws, perm_out, key_out, stream);
}

int sched_best(const void *ws, uint16_t *perm_out, int64_t *key_out, hipStream_t stream) {
  if (!ws || !perm_out || !key_out) return SCHED_EINVAL;
  sa::best_copy_kernel<<<1, 256, 0, stream>>>(static_cast<const unsigned char *>(ws), perm_out, key_out);
  HIP_TRY(hipGetLastError());
  return SCHED_OK;
}

int sched_chains(const void *ws, int64_t *per_chain, uint16_t *cur_perms, uint16_t *best_perms, hipStream_t stream) {
  if (!ws || !per_chain) return SCHED_EINVAL;
  sa::chains_copy_kernel<<<256, 256, 0, stream>>>(static_cast<const unsigned char *>(ws), per_chain, cur_perms,
                                                  best_perms);
  HIP_TRY(hipGetLastError());
  return SCHED_OK;
}

int sched_start_info(const void *ws, uint16_t *start_out, int64_t *info_out, hipStream_t stream) {
  if (!ws || !start_out || !info_out) return SCHED_EINVAL;
  sa::start_copy_kernel<<<1, 256, 0, stream>>>(static_cast<const unsigned char *>(ws), start_out, info_out);
  HIP_TRY(hipGetLastError());
  return SCHED_OK;
}

int sched_gen_perms(uint64_t seed, int32_t n, int64_t row0, int64_t k, uint16_t *perms, hipStream_t stream) {
  if (n < 1 || n > SCHED_MAX_N || row0 < 0 || k < 0 || row0 + k > (int64_t)UINT32_MAX + 1) return SCHED_EINVAL;
  if (k == 0) return SCHED_OK;
  if (!perms) return SCHED_EINVAL;
  const int64_t grid = (k + 255) / 256;
  sa::shuffle_kernel<<<(unsigned)grid, 256, 0, stream>>>((uint32_t)seed, (uint32_t)(seed >> 32), n, row0, k, perms);
  HIP_TRY(hipGetLastError());
  return SCHED_OK;
}

int sched_eval_batches(const sched_queue_t *queue, const sched_model_t *model, const uint16_t *perms,
                       const uint8_t *starts, int64_t k, int64_t *out, int64_t *detail, hipStream_t stream) {
  if (k < 0) return SCHED_EINVAL;
  int rc = check_queue(queue);
  if (rc) return rc;
  if ((rc = check_model(model, queue->n))) return rc;
  if (model->policy == SCHED_CONTINUOUS) return SCHED_EINVAL;
  if (k > 0 && (!perms || !starts || !out)) return SCHED_EINVAL;
  if (k == 0) return SCHED_OK;
  const int n = queue->n;
  const sa::QueuePtrs qp = dev_queue(queue);
  const size_t pb = ((size_t)n * 2 + 15) & ~size_t(15), fb = ((size_t)n + 15) & ~size_t(15);
  const size_t lds = (((size_t)n * 16 + 15) & ~size_t(15)) + 4 * (pb + fb + 64 * 16 + 32 * 4);
  const int grid = (int)std::min<int64_t>((k + 3) / 4, 256 * 32);
  Candidates<sa::DevModel> c;
  // one kernel: the windowed replay, the 32-bit pair costs and the 32-bit timeline are taken
  // where they hold
  c.add(0u, sa::kFlagWindows | kSN | kT32, [=](const sa::DevModel &d) {
    if (detail)
      sa::eval_sized_kernel<true><<<grid, 256, lds, stream>>>(d, qp, perms, starts, k, out, detail);
    else
      sa::eval_sized_kernel<false><<<grid, 256, lds, stream>>>(d, qp, perms, starts, k, out, nullptr);
    return hipGetLastError();
  });
  return c.run(dev_model(model, n));
}

int sched_starts(const void *ws, uint8_t *cur_starts, uint8_t *best_starts, uint8_t *winner_starts,
                 hipStream_t stream) {
  if (!ws || (!cur_starts && !best_starts && !winner_starts)) return SCHED_EINVAL;
  sa::starts_copy_kernel<<<256, 256, 0, stream>>>(static_cast<const unsigned char *>(ws), cur_starts, best_starts,
                                                  winner_starts);
  HIP_TRY(hipGetLastError());
  return SCHED_OK;
}

int sched_status(const void *ws, int64_t *out, hipStream_t stream) {
  if (!ws || !out) return SCHED_EINVAL;
  sa::status_copy_kernel<<<1, 1, 0, stream>>>(static_cast<const unsigned char *>(ws), out);
  HIP_TRY(hipGetLastError());
  return SCHED_OK;
}

int sched_assign(const sched_queue_t *queue, int32_t instances, const int64_t *capacity, int32_t *inst_out,
                 hipStream_t stream) {
  int rc = check_queue(queue);
  if (rc) return rc;
  if (instances < 1 || instances > SCHED_MAX_INSTANCES || !capacity || !inst_out) return SCHED_EINVAL;
  sa::assign_kernel<<<1, 64, 0, stream>>>(dev_queue(queue), queue->n, instances, capacity, inst_out);
  HIP_TRY(hipGetLastError());
  return SCHED_OK;
}

size_t sched_ws_bytes_multi(int32_t n, int32_t instances, int32_t chains) {
  if (n < 1 || n > SCHED_MAX_N || instances < 1 || instances > SCHED_MAX_INSTANCES || chains < 1) return 0;
  return sa::mws_total(n, instances, chains);
}

int sched_anneal_multi(const sched_queue_t *queue, const sched_model_t *model, const sched_search_t *search,
                       const int32_t *inst_of, int32_t instances, int32_t chains, int32_t iters, double T0,
                       double alpha, uint64_t seed, void *ws, size_t ws_bytes, hipStream_t stream) {
  int rc = check_queue(queue);
  if (rc) return rc;
  if (instances < 1 || instances > SCHED_MAX_INSTANCES || !inst_of) return SCHED_EINVAL;
  if ((rc = check_chain_args(chains, iters, T0, alpha))) return rc;
  sa::SearchParams srch;
  if ((rc = check_search(search, srch))) return rc;
  if ((rc = check_model(model, queue->n))) return rc;
  if (model->policy == SCHED_STATIC_SEARCH) return SCHED_EINVAL;
  if (srch.objective == SCHED_OBJ_RATIO && model->p0 + model->d0 + model->d1 < 1) return SCHED_EINVAL;
  const int n = queue->n;
  if (!ws || (reinterpret_cast<uintptr_t>(ws) & 255u)) return SCHED_EINVAL;
  if (ws_bytes < sched_ws_bytes_multi(n, instances, chains)) return SCHED_ENOSPC;
  const sa::DevModel dm = dev_model(model, n, 2, srch.objective == SCHED_OBJ_RATIO);
  unsigned char *w = static_cast<unsigned char *>(ws);
  const MultiArgs a{n, instances, chains, iters, T0, alpha, (uint32_t)seed, (uint32_t)(seed >> 32),
                    model->swap_threshold, srch, w, stream};
  Candidates<sa::DevModel> c;
  if (srch.objective)
    add_multi<1>(c, model, a);
  else
    add_multi<0>(c, model, a);
  const sa::QueuePtrs qp = dev_queue(queue);
  sa::multi_plan_kernel<<<1, 1024, 0, stream>>>(c.checker(dm, 0u), qp, inst_of, instances, chains, iters,
                                                (int64_t)sa::mws_slot_bytes(n, chains), w);
  HIP_TRY(hipGetLastError());
  sa::gather_kernel<<<instances, 1024, 0, stream>>>(qp, n, inst_of, chains, instances, w);
  HIP_TRY(hipGetLastError());
  sa::multi_start_kernel<<<instances, 1024, 0, stream>>>(c.checker(dm, kMultiFlags), n, instances, chains, iters,
                                                         model->t_ref_us, srch, w);
  HIP_TRY(hipGetLastError());
  if ((rc = c.run(dm))) return rc;
  sa::multi_reduce_kernel<<<instances, 1024, 0, stream>>>(n, instances, chains, w);
  HIP_TRY(hipGetLastError());
  return SCHED_OK;
}

void *sched_multi_instance_ws(void *ws, int32_t n, int32_t instances, int32_t chains, int32_t instance) {
  if (!ws || n < 1 || n > SCHED_MAX_N || instances < 1 || instances > SCHED_MAX_INSTANCES || chains < 1 ||
      instance < 0 || instance >= instances)
    return nullptr;
  return static_cast<unsigned char *>(ws) + sa::mws_off_slot(n, instances, chains, instance);
}

int sched_multi_best(const void *ws, int32_t instances, uint16_t *orders, int64_t *keys, int32_t *counts,
                     hipStream_t stream) {
  if (!ws || !orders || instances < 1 || instances > SCHED_MAX_INSTANCES) return SCHED_EINVAL;
  sa::multi_best_kernel<<<instances, 256, 0, stream>>>(static_cast<const unsigned char *>(ws), orders, keys, counts);
  HIP_TRY(hipGetLastError());
  return SCHED_OK;
}

int sched_eval_fit(const sched_queue_t *queue, const sched_fit_model_t *fit, const uint32_t *tpot_thr,
                   const uint16_t *perms, const uint8_t *starts, int64_t k, int64_t *out, int64_t *detail,
                   hipStream_t stream) {
  if (k < 0) return SCHED_EINVAL;
  int rc = check_queue(queue);
  if (rc) return rc;
  if ((rc = check_fit(fit))) return rc;
  if (k > 0 && (!perms || !out)) return SCHED_EINVAL;
  if (k == 0) return SCHED_OK;
  const int n = queue->n;
  const sa::QueuePtrs qp = dev_queue(queue);
  const size_t pb = ((size_t)n * 2 + 15) & ~size_t(15), fb = ((size_t)n + 15) & ~size_t(15);
  const size_t lds = (((size_t)n * 16 + 15) & ~size_t(15)) + 4 * (pb + fb + 32 * 4);
  const int grid = (int)std::min<int64_t>((k + 3) / 4, 256 * 32);
  Candidates<sa::DevFit> c;
  c.add(0u, sa::kFlagFitWindows, [=](const sa::DevFit &d) {
    if (detail)
      sa::eval_fit_kernel<true><<<grid, 256, lds, stream>>>(d, qp, tpot_thr, perms, starts, k, out, detail);
    else
      sa::eval_fit_kernel<false><<<grid, 256, lds, stream>>>(d, qp, tpot_thr, perms, starts, k, out, nullptr);
    return hipGetLastError();
  });
  return c.run(dev_fit(fit, n, tpot_thr ? 3 : 2, 0));
}

int sched_anneal_fit(const sched_queue_t *queue, const sched_fit_model_t *fit, const uint32_t *tpot_thr,
                     const sched_search_t *search, int32_t chains, int32_t iters, double T0, double alpha,
                     uint64_t seed, void *ws, size_t ws_bytes, hipStream_t stream) {
  int rc = check_queue(queue);
  if (rc) return rc;
  if ((rc = check_chain_args(chains, iters, T0, alpha))) return rc;
  sa::SearchParams srch;
  if ((rc = check_search(search, srch))) return rc;
  if ((rc = check_fit(fit))) return rc;
  if (srch.objective == SCHED_OBJ_RATIO && fit->dp + fit->dd < 1) return SCHED_EINVAL;  // positive latencies
  if (!ws || (reinterpret_cast<uintptr_t>(ws) & 255u)) return SCHED_EINVAL;
  if (ws_bytes < sched_ws_bytes(queue->n, chains)) return SCHED_ENOSPC;
  const int n = queue->n;
  const sa::DevFit df = dev_fit(fit, n, tpot_thr ? 3 : 2, srch.objective == SCHED_OBJ_RATIO);
  unsigned char *w = static_cast<unsigned char *>(ws);
  const sa::QueuePtrs qp = dev_queue(queue);
  const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
  const uint64_t st = fit->swap_threshold;
  constexpr uint32_t kFitFlags = sa::kFlagFitWindows | sa::kFlagFitMember32;
  Candidates<sa::DevFit> c;
  if (n <= 64) {
    // small queue: order, request fields and layout in registers, no LDS (the windowed
    // replay's keys must fit)
    const int waves = reg_waves(chains), grid = (chains + waves - 1) / waves;
    c.add(sa::kFlagFitWindows, kFitFlags, [=](const sa::DevFit &d) {
      if (srch.objective)
        sa::anneal_reg_fit_kernel<1><<<grid, waves * 64, 0, stream>>>(d, qp, tpot_thr, chains, iters, T0, alpha, k0,
                                                                      k1, st, srch, w);
      else
        sa::anneal_reg_fit_kernel<0><<<grid, waves * 64, 0, stream>>>(d, qp, tpot_thr, chains, iters, T0, alpha, k0,
                                                                      k1, st, srch, w);
      return hipGetLastError();
    });
  }
  const size_t pb = ((size_t)n * 2 + 15) & ~size_t(15), fb = ((size_t)n + 15) & ~size_t(15);
  const size_t lds = (((size_t)n * 16 + 15) & ~size_t(15)) + 4 * (2 * pb + 2 * fb);
  const int grid = (chains + 3) / 4;
  c.add(0u, kFitFlags, [=](const sa::DevFit &d) {
    if (srch.objective)
      sa::anneal_fit_kernel<1><<<grid, 256, lds, stream>>>(d, qp, tpot_thr, chains, iters, T0, alpha, k0, k1, st, srch,
                                                           w);
    else
      sa::anneal_fit_kernel<0><<<grid, 256, lds, stream>>>(d, qp, tpot_thr, chains, iters, T0, alpha, k0, k1, st, srch,
                                                           w);
    return hipGetLastError();
  });
  sa::start_fit_kernel<<<1, 1024, 0, stream>>>(c.checker(df, kFitFlags), qp, tpot_thr, chains, iters, fit->t_ref, srch,
                                               w);
  HIP_TRY(hipGetLastError());
  if ((rc = c.run(df))) return rc;
  sa::reduce_kernel<<<1, 1024, 0, stream>>>(w);
  HIP_TRY(hipGetLastError());
  return SCHED_OK;
}

int sched_accept_check(int32_t rule, int64_t k, const int64_t *a, const int64_t *b, const uint64_t *c,
                       const uint64_t *d, const double *T, const uint32_t *w3, uint8_t *out, hipStream_t stream) {
  if ((rule != 0 && rule != 1) || k < 0) return SCHED_EINVAL;
  if (k == 0) return SCHED_OK;
  if (!a || !b || !T || !w3 || !out || (rule == 1 && (!c || !d))) return SCHED_EINVAL;
  const int grid = (int)std::min<int64_t>((k + 255) / 256, 4096);
  sa::accept_check_kernel<<<grid, 256, 0, stream>>>(rule, k, a, b, c, d, T, w3, out);
  HIP_TRY(hipGetLastError());
  return SCHED_OK;
}

int32_t sched_levels(double T0, double T_thres, double tau) {
  if (!(T0 > 0.0) || !std::isfinite(T0) || !(T_thres > 0.0) || !std::isfinite(T_thres) || !(tau > 0.0) ||
      !(tau < 1.0))
    return SCHED_EINVAL;
  int32_t levels = 0;
  double T = T0;
  do {
    ++levels;
    T = T * tau;
  } while (T >= T_thres && levels < (1 << 30));
  return levels;
}

const char *sched_strerror(int code) {
  switch (code) {
    case SCHED_OK: return "ok";
    case SCHED_EINVAL: return "invalid argument, size, model parameter or queue entry";
    case SCHED_ENOSPC:
      return "workspace smaller than sched_ws_bytes(n, chains) (for sched_anneal_noalloc: that size exceeds "
             "SCHED_NOALLOC_MAX_BYTES)";
    case SCHED_ERANGE: return "queue and model could overflow the int64 clock or objective";
    case SCHED_EHIP: return g_hip_msg.empty() ? "HIP runtime error" : g_hip_msg.c_str();
    default: return "unknown error code";
  }
}

}  // extern "C"
