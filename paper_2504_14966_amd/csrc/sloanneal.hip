// C-ABI of the annealing library (declared in include/sloanneal.h): argument and queue
// validation, int64 range pre-checks, workspace sizing and kernel launches on the caller's
// stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/sloanneal.h"
#include "kernels.h"
#include "anneal_static.h"
#include "anneal_wave.h"
#include "anneal_sized.h"
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

struct HostQueue {
  std::vector<uint16_t> in_len, out_len;
  std::vector<uint8_t> kind;
  std::vector<uint32_t> thr;
};

int check_model(const sched_model_t *m, int n) {
  if (!m) return SCHED_EINVAL;
  if (m->max_batch < 1 || m->max_batch > SCHED_MAX_BATCH) return SCHED_EINVAL;
  if (m->policy != SCHED_STATIC && m->policy != SCHED_CONTINUOUS && m->policy != SCHED_STATIC_SEARCH) return SCHED_EINVAL;
  if (m->p0 < 0 || m->p1 < 0 || m->d0 < 0 || m->d1 < 0 || m->d2 < 0 || m->t_ref_us < 0) return SCHED_EINVAL;
  if (m->swap_threshold > (1ull << 32)) return SCHED_EINVAL;
  (void)n;
  return SCHED_OK;
}

// Reads the queue back (one stream synchronisation) and validates every entry (kinds up to
// max_kind).
int fetch_queue(const sched_queue_t *q, hipStream_t stream, HostQueue &h, int max_kind = 2) {
  if (!q || q->n < 1 || q->n > SCHED_MAX_N) return SCHED_EINVAL;
  if (!q->in_len || !q->out_len || !q->kind || !q->thr_us) return SCHED_EINVAL;
  const size_t n = (size_t)q->n;
  h.in_len.resize(n);
  h.out_len.resize(n);
  h.kind.resize(n);
  h.thr.resize(n);
  HIP_TRY(hipMemcpyAsync(h.in_len.data(), q->in_len, n * 2, hipMemcpyDeviceToHost, stream));
  HIP_TRY(hipMemcpyAsync(h.out_len.data(), q->out_len, n * 2, hipMemcpyDeviceToHost, stream));
  HIP_TRY(hipMemcpyAsync(h.kind.data(), q->kind, n, hipMemcpyDeviceToHost, stream));
  HIP_TRY(hipMemcpyAsync(h.thr.data(), q->thr_us, n * 4, hipMemcpyDeviceToHost, stream));
  HIP_TRY(hipStreamSynchronize(stream));
  for (size_t r = 0; r < n; ++r) {
    if (h.out_len[r] < 1 || h.kind[r] > max_kind || h.thr[r] > SCHED_THR_MAX) return SCHED_EINVAL;
  }
  return SCHED_OK;
}

// Worst-case clock: every request's prefill plus, per request, its decode iterations at
// the largest possible step cost. The sum over requests and the Metropolis delta
// (|dn| <= n times t_ref) must stay below 2^62.
// Bound on the timeline of any order and any batch layout: every prefill, plus per decode
// step (at most the sum of output lengths) the cost of a full batch of the longest contexts.
long double timeline_bound(const HostQueue &h, const sched_model_t *m, int n) {
  long double max_lin = 0, max_lout = 0, sum_lout = 0, pre = 0;
  for (int r = 0; r < n; ++r) {
    max_lin = std::max<long double>(max_lin, h.in_len[r]);
    max_lout = std::max<long double>(max_lout, h.out_len[r]);
    sum_lout += h.out_len[r];
    pre += (long double)m->p0 + (long double)m->p1 * h.in_len[r];
  }
  const long double b = std::min(n, m->max_batch);
  const long double step = (long double)m->d0 + (long double)m->d1 * b + (long double)m->d2 * b * (max_lin + max_lout);
  return pre + sum_lout * step;
}

int range_check(const HostQueue &h, const sched_model_t *m, int n) {
  const long double lim = std::ldexp(1.0L, 62);
  const long double clock = timeline_bound(h, m, n);
  const long double tsum = clock * n;
  const long double tref = m->t_ref_us > 0 ? (long double)m->t_ref_us : tsum;
  if (!(tsum < lim) || !(tref * (n + 1) + tsum < lim)) return SCHED_ERANGE;
  return SCHED_OK;
}

// The fitted model: every coefficient >= 0, batches of 1 .. 64. A member's time is largest
// at the largest batch, and a batch lasts at most the sum of its members' times, so the
// timeline ends before the sum over requests of their time in a batch of min(n, B); the sum
// of latencies, the Metropolis delta and (for the ratio) the cross products stay below 2^62.
int check_fit(const sched_fit_model_t *f) {
  if (!f || f->max_batch < 1 || f->max_batch > SCHED_MAX_BATCH) return SCHED_EINVAL;
  if (f->policy != SCHED_STATIC && f->policy != SCHED_STATIC_SEARCH) return SCHED_EINVAL;
  if (f->ap < 0 || f->bp < 0 || f->cp < 0 || f->dp < 0 || f->ad < 0 || f->bd < 0 || f->cd < 0 || f->dd < 0 ||
      f->t_ref < 0 || f->swap_threshold > (1ull << 32))
    return SCHED_EINVAL;
  return SCHED_OK;
}

// Sum over requests of their time in a batch of min(n, B): a member's time grows with its
// batch size, and a batch lasts at most the sum of its members' times, so this bounds the
// timeline and every member's time.
long double fit_timeline_bound(const HostQueue &h, const sched_fit_model_t *f, int n) {
  const long double b = std::min(n, f->max_batch);
  long double end = 0;
  for (int r = 0; r < n; ++r) {
    const long double l = h.in_len[r], L = h.out_len[r];
    end += (long double)f->ap * b * l + (long double)f->bp * b + (long double)f->cp * l + (long double)f->dp +
           L * ((long double)f->bd * b + (long double)f->dd) +
           ((long double)f->ad * b + (long double)f->cd) * (L * l + L * (L + 1) / 2);
  }
  return end;
}

int fit_range_check(const HostQueue &h, const sched_fit_model_t *f, int n, bool ratio) {
  const long double end = fit_timeline_bound(h, f, n);
  const long double tsum = end * n, lim = std::ldexp(1.0L, 62);
  const long double tref = f->t_ref > 0 ? (long double)f->t_ref : tsum;
  if (!(tsum < lim) || !(tref * (n + 1) + tsum < lim)) return SCHED_ERANGE;
  if (ratio && !(tsum * (n + 1) < lim)) return SCHED_ERANGE;
  return SCHED_OK;
}

// The largest time of one request in any batch (times grow with the batch size).
long double fit_member_bound(const HostQueue &h, const sched_fit_model_t *f, int n) {
  const long double b = std::min(n, f->max_batch);
  long double mx = 0;
  for (int r = 0; r < n; ++r) {
    const long double l = h.in_len[r], L = h.out_len[r];
    mx = std::max(mx, (long double)f->ap * b * l + (long double)f->bp * b + (long double)f->cp * l +
                          (long double)f->dp + L * ((long double)f->bd * b + (long double)f->dd) +
                          ((long double)f->ad * b + (long double)f->cd) * (L * l + L * (L + 1) / 2));
  }
  return mx;
}

// win: the windowed replay's keys hold every member's time (below 2^57 with margin);
// m32: every member's time fits 32 bits
sa::DevFit dev_fit(const sched_fit_model_t *f, int n, bool win, bool m32 = false) {
  return sa::DevFit{n, f->max_batch, f->policy, 0, (uint64_t)f->ap, (uint64_t)f->bp, (uint64_t)f->cp,
                    (uint64_t)f->dp, (uint64_t)f->ad, (uint64_t)f->bd, (uint64_t)f->cd, (uint64_t)f->dd,
                    win ? 1u : 0u, m32 ? 1u : 0u, (1ull << 32) / (uint64_t)f->max_batch + 1};
}

// The ratio objective compares n1 t2 with n2 t1 and forms n' t - n t' in int64: the
// worst-case total latency times (n + 1) stays below 2^62.
int ratio_range_check(const HostQueue &h, const sched_model_t *m, int n) {
  long double max_lin = 0, max_lout = 0, sum_lout = 0, pre = 0;
  for (int r = 0; r < n; ++r) {
    max_lin = std::max<long double>(max_lin, h.in_len[r]);
    max_lout = std::max<long double>(max_lout, h.out_len[r]);
    sum_lout += h.out_len[r];
    pre += (long double)m->p0 + (long double)m->p1 * h.in_len[r];
  }
  const long double b = std::min(n, m->max_batch);
  const long double step = (long double)m->d0 + (long double)m->d1 * b + (long double)m->d2 * b * (max_lin + max_lout);
  const long double tsum = (pre + sum_lout * step) * n;
  return tsum * (n + 1) < std::ldexp(1.0L, 62) ? SCHED_OK : SCHED_ERANGE;
}

// The continuous event loop's 32-bit arithmetic: group prefill sums, the context sum C of
// the running requests, d0 + d1 b + d2 C and d2 b all stay below 2^32.
bool prefill_narrow(const HostQueue &h, const sched_model_t *m, int n) {
  long double lmax = 0, Lmax = 0;
  for (int r = 0; r < n; ++r) {
    lmax = std::max<long double>(lmax, h.in_len[r]);
    Lmax = std::max<long double>(Lmax, h.out_len[r]);
  }
  const long double b = std::min(n, m->max_batch), two32 = 4294967296.0L;
  const long double pf = (long double)m->p0 + (long double)m->p1 * lmax;
  const long double cmax = b * (lmax + Lmax);
  const long double x = (long double)m->d0 + (long double)m->d1 * b + (long double)m->d2 * cmax;
  return pf * b < two32 && cmax < two32 && x < two32 && (long double)m->d2 * b < two32;
}

// List scheduling packs (finish step << 10 | position) into 32 bits and keeps prefix
// sums of prefill costs in 32 bits: the total of all output lengths stays below 2^22 and
// the total prefill below 2^32.
bool list_sched_ok(const HostQueue &h, const sched_model_t *m, int n) {
  long double lsum = 0, pfsum = 0;
  for (int r = 0; r < n; ++r) {
    lsum += h.out_len[r];
    pfsum += (long double)m->p0 + (long double)m->p1 * h.in_len[r];
  }
  return n <= 1024 && lsum < 4194304.0L && pfsum < 4294967296.0L;
}

// Continuous admission: every time on the timeline is at most the sum of the prefills plus
// the decode steps' costs, sum over steps of d0 + d1 b + d2 C. There are at most sum(l_out)
// steps, the b terms add up to sum(l_out) and the C terms to sum(l_out l_in + l_out (l_out
// + 1) / 2), whatever the order.
bool timeline_narrow(const HostQueue &h, const sched_model_t *m, int n) {
  long double pf = 0, L = 0, ctx = 0;
  for (int r = 0; r < n; ++r) {
    const long double lo = h.out_len[r], li = h.in_len[r];
    pf += (long double)m->p0 + (long double)m->p1 * li;
    L += lo;
    ctx += lo * li + lo * (lo + 1) / 2;
  }
  return pf + ((long double)m->d0 + (long double)m->d1) * L + (long double)m->d2 * ctx < 4294967296.0L;
}

sa::DevModel dev_model(const sched_model_t *m, int n, bool narrow_prefill, bool list_sched = false,
                       bool narrow_time = false, bool windows = false, bool static_narrow_w = false) {
  sa::DevModel d;
  d.n = n;
  d.B = m->max_batch;
  d.policy = m->policy;
  d.flags = (narrow_prefill ? sa::kFlagNarrowPrefill : 0) | (narrow_prefill && list_sched ? sa::kFlagListSched : 0) |
            (narrow_prefill && list_sched && narrow_time ? sa::kFlagNarrowTime : 0) | (windows ? sa::kFlagWindows : 0) |
            (static_narrow_w ? sa::kFlagStaticNarrow : 0);
  d.p0 = (uint64_t)m->p0;
  d.p1 = (uint64_t)m->p1;
  d.d0 = (uint64_t)m->d0;
  d.d1 = (uint64_t)m->d1;
  d.d2 = (uint64_t)m->d2;
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

// The delta kernel keeps finish offsets, prefills, slacks and doubled pair costs in 32
// bits and forms each doubled pair cost mu * (e + d2 * mu), e = 2 (d1 + d2 l_in) + d2, with
// 24-bit multiplies. Every finish offset is at most B * max prefill + L_max * d0 + B *
// (d1 * L_max + d2 * (l_max * L_max + L_max (L_max + 1) / 2)).
bool static_narrow(const HostQueue &h, const sched_model_t *m, int n) {
  long double lmax = 0, Lmax = 0;
  for (int r = 0; r < n; ++r) {
    lmax = std::max<long double>(lmax, h.in_len[r]);
    Lmax = std::max<long double>(Lmax, h.out_len[r]);
  }
  const long double b = std::min(n, m->max_batch);
  const long double pf = (long double)m->p0 + (long double)m->p1 * lmax;
  const long double fmax = b * pf + Lmax * m->d0 +
                           b * ((long double)m->d1 * Lmax + (long double)m->d2 * (lmax * Lmax + Lmax * (Lmax + 1) / 2));
  const long double emax = 2.0L * ((long double)m->d1 + (long double)m->d2 * lmax) + m->d2;
  const long double inner = emax + (long double)m->d2 * Lmax;
  const long double two24 = 16777216.0L, two32 = 4294967296.0L;
  return fmax < two32 - 1 && inner < two24 && (long double)m->d2 < two24 && b * Lmax * inner < two32 &&
         (long double)m->d0 < two24;
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

template <int LG, int OBJ>
hipError_t launch_static(int waves, size_t lds, const sa::DevModel &dm, const sa::StaticParams &sp,
                         const sa::QueuePtrs &q, int chains, int iters, double T0, double alpha, uint64_t seed,
                         uint64_t swap_thr, const sa::SearchParams &srch, unsigned char *w, hipStream_t stream) {
  if (lds > 65536) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(&sa::anneal_static_kernel<LG, OBJ>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  const int grid = (chains + waves - 1) / waves;
  sa::anneal_static_kernel<LG, OBJ><<<grid, waves * 64, lds, stream>>>(dm, sp, q, chains, iters, T0, alpha,
                                                                       (uint32_t)seed, (uint32_t)(seed >> 32), swap_thr,
                                                                       srch, w);
  return hipGetLastError();
}

// The batch-size search's delta kernel keeps finish offsets, prefills and pair costs as the
// fixed-size delta kernel does (static_narrow) and every time on the timeline in 32 bits:
// whatever the layout, the timeline ends within the sum of all prefills plus, per decode
// iteration, d0 + d1 b + d2 C; there are at most sum(l_out) iterations, the b terms add up
// to sum(l_out) and the C terms to sum(l_out l_in + l_out (l_out + 1) / 2).
bool sized_narrow(const HostQueue &h, const sched_model_t *m, int n) {
  long double pf = 0, L = 0, ctx = 0;
  for (int r = 0; r < n; ++r) {
    const long double lo = h.out_len[r], li = h.in_len[r];
    pf += (long double)m->p0 + (long double)m->p1 * li;
    L += lo;
    ctx += lo * li + lo * (lo + 1) / 2;
  }
  const long double end = pf + ((long double)m->d0 + (long double)m->d1) * L + (long double)m->d2 * ctx;
  return static_narrow(h, m, n) && end < 4294967295.0L - 1.0L;
}

size_t sized_chain_lds(int n) {
  const size_t pb = ((size_t)n * 2 + 15) & ~size_t(15), fb = ((size_t)n + 15) & ~size_t(15);
  const size_t ub = ((size_t)n * 4 + 15) & ~size_t(15), sb = ((size_t)(n + 1) * 4 + 15) & ~size_t(15);
  return pb + fb + 2 * ub + sb;
}

// Joint order / batch-size search: the delta kernel when the widths allow (as many chains
// per workgroup as spread the chains over every CU, at most 16 and at most what the LDS
// holds), else the full-replay kernel, four chains per workgroup.
template <int OBJ>
int launch_sized(const HostQueue &h, const sched_model_t *model, const sa::DevModel &dm, const sched_queue_t *queue,
                 int chains, int iters, double T0, double alpha, uint64_t seed, const sa::SearchParams &srch,
                 unsigned char *w, hipStream_t stream) {
  const int n = dm.n;
  if (sa::reg_sized_fits(n) && static_narrow(h, model, n)) {
    // small queue: the order, every request field and the layout in registers, no LDS
    const int cus = std::max(1, cu_count());
    const int waves = chains >= 4 * cus ? 4 : (chains >= 2 * cus ? 2 : 1);
    const int grid = (chains + waves - 1) / waves;
    sa::DevModel dr = dm;  // the whole timeline in 32 bits: plain prefix sums
    if (sized_narrow(h, model, n)) dr.flags |= sa::kFlagTime32;
    sa::anneal_reg_sized_kernel<OBJ><<<grid, waves * 64, 0, stream>>>(dr, dev_queue(queue), chains, iters, T0, alpha,
                                                                      (uint32_t)seed, (uint32_t)(seed >> 32), srch, w);
    HIP_TRY(hipGetLastError());
    return SCHED_OK;
  }
  if (sized_narrow(h, model, n)) {
    const size_t soa = (size_t)(n + 1) * 16, per = sized_chain_lds(n);
    const int lim = max_lds_per_block(), cus = std::max(1, cu_count());
    int waves = 1;
    while (waves < 16 && (int64_t)waves * cus < chains) waves <<= 1;
    while (waves > 1 && soa + per * waves > (size_t)lim) waves >>= 1;
    if (soa + per * waves <= (size_t)lim) {
      const size_t lds = soa + per * waves;
      if (lds > 65536)
        HIP_TRY(hipFuncSetAttribute(reinterpret_cast<const void *>(&sa::anneal_sized_kernel<OBJ>),
                                    hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds));
      const sa::StaticParams sp{(uint32_t)model->d0, (uint32_t)model->d2, (1ull << 32) / (uint64_t)model->max_batch + 1};
      const int grid = (chains + waves - 1) / waves;
      sa::anneal_sized_kernel<OBJ><<<grid, waves * 64, lds, stream>>>(dm, sp, dev_queue(queue), chains, iters, T0,
                                                                      alpha, (uint32_t)seed, (uint32_t)(seed >> 32),
                                                                      srch, w);
      HIP_TRY(hipGetLastError());
      return SCHED_OK;
    }
  }
  const size_t pb = ((size_t)n * 2 + 15) & ~size_t(15), fb = ((size_t)n + 15) & ~size_t(15);
  const size_t lds = (((size_t)n * 16 + 15) & ~size_t(15)) + 4 * (2 * pb + 2 * fb + 64 * 16);
  const int grid = (chains + 3) / 4;
  sa::anneal_sized_generic_kernel<OBJ><<<grid, 256, lds, stream>>>(dm, dev_queue(queue), chains, iters, T0, alpha,
                                                                   (uint32_t)seed, (uint32_t)(seed >> 32), srch, w);
  HIP_TRY(hipGetLastError());
  return SCHED_OK;
}

size_t anneal_lds_bytes(int n) {
  const size_t per_wave = ((size_t)n * 2 + 15) / 16 * 16 * 2 + 64 * 16;
  return ((size_t)n * 16 + 15) / 16 * 16 + per_wave * sa::kWavesPerBlock;
}

// Every chain of one sched_anneal: the kernel for the policy and the widths the queue and
// model allow (see the checks above), objective OBJ.
template <int OBJ>
int launch_chains(const HostQueue &h, const sched_model_t *model, const sa::DevModel &dm, const sched_queue_t *queue,
                  int chains, int iters, double T0, double alpha, uint64_t seed, const sa::SearchParams &srch,
                  unsigned char *w, hipStream_t stream) {
  const int n = dm.n;
  int rc = SCHED_OK;
  bool done = false;
  if (model->policy == SCHED_STATIC_SEARCH) {
    if ((rc = launch_sized<OBJ>(h, model, dm, queue, chains, iters, T0, alpha, seed, srch, w, stream))) return rc;
    done = true;
  }
  if (!done && model->policy == SCHED_STATIC && sa::reg_kernel_fits(n, model->max_batch) &&
      static_narrow(h, model, n)) {
    // small queue: the order and every request field in registers, no LDS; four chains per
    // workgroup, or fewer so that the chains spread over every CU
    const int cus = std::max(1, cu_count());
    const int waves = chains >= 4 * cus ? 4 : (chains >= 2 * cus ? 2 : 1);
    const int grid = (chains + waves - 1) / waves;
    const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
    const sa::QueuePtrs qp = dev_queue(queue);
    const uint64_t st = model->swap_threshold;
    sa::DevModel dr = dm;  // every time in 32 bits: the 32-bit start scan and latency sum
    if (sized_narrow(h, model, n)) dr.flags |= sa::kFlagTime32;
    switch (model->max_batch) {
      case 1: sa::anneal_reg_kernel<0, OBJ><<<grid, waves * 64, 0, stream>>>(dr, qp, chains, iters, T0, alpha, k0, k1, st, srch, w); break;
      case 2: sa::anneal_reg_kernel<1, OBJ><<<grid, waves * 64, 0, stream>>>(dr, qp, chains, iters, T0, alpha, k0, k1, st, srch, w); break;
      case 4: sa::anneal_reg_kernel<2, OBJ><<<grid, waves * 64, 0, stream>>>(dr, qp, chains, iters, T0, alpha, k0, k1, st, srch, w); break;
      case 8: sa::anneal_reg_kernel<3, OBJ><<<grid, waves * 64, 0, stream>>>(dr, qp, chains, iters, T0, alpha, k0, k1, st, srch, w); break;
      default: sa::anneal_reg_kernel<4, OBJ><<<grid, waves * 64, 0, stream>>>(dr, qp, chains, iters, T0, alpha, k0, k1, st, srch, w); break;
    }
    HIP_TRY(hipGetLastError());
    done = true;
  }
  if (!done && model->policy == SCHED_STATIC && sa::reg_parts(n, model->max_batch) > 1 &&
      static_narrow(h, model, n)) {
    // 65 to 192 requests: two or three positions per lane, still no LDS
    const int cus = std::max(1, cu_count());
    const int waves = chains >= 4 * cus ? 4 : (chains >= 2 * cus ? 2 : 1);
    const int grid = (chains + waves - 1) / waves;
    const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
    const sa::QueuePtrs qp = dev_queue(queue);
    const uint64_t st = model->swap_threshold;
    sa::DevModel dr = dm;
    if (sized_narrow(h, model, n)) dr.flags |= sa::kFlagTime32;
    switch (model->max_batch) {
      case 1: sa::anneal_reg_h_kernel<0, OBJ><<<grid, waves * 64, 0, stream>>>(dr, qp, chains, iters, T0, alpha, k0, k1, st, srch, w); break;
      case 2: sa::anneal_reg_h_kernel<1, OBJ><<<grid, waves * 64, 0, stream>>>(dr, qp, chains, iters, T0, alpha, k0, k1, st, srch, w); break;
      case 4: sa::anneal_reg_h_kernel<2, OBJ><<<grid, waves * 64, 0, stream>>>(dr, qp, chains, iters, T0, alpha, k0, k1, st, srch, w); break;
      case 8: sa::anneal_reg_h_kernel<3, OBJ><<<grid, waves * 64, 0, stream>>>(dr, qp, chains, iters, T0, alpha, k0, k1, st, srch, w); break;
      default: sa::anneal_reg_h_kernel<4, OBJ><<<grid, waves * 64, 0, stream>>>(dr, qp, chains, iters, T0, alpha, k0, k1, st, srch, w); break;
    }
    HIP_TRY(hipGetLastError());
    done = true;
  }
  if (!done && model->policy == SCHED_STATIC && static_narrow(h, model, n)) {
    // chains per workgroup: enough to spread the chains over every CU, at most 16 and
    // at most what the LDS holds
    int lg = 0;
    while ((1 << lg) < model->max_batch) ++lg;
    // a batch of more than 32 requests fills a wave: the lane-per-batch kernel
    const bool wave_kernel = lg == 6;
    const size_t soa = (size_t)(n + 1) * 16;
    const size_t per = wave_kernel ? wave_chain_lds(n, model->max_batch) : static_wave_lds(n, model->max_batch);
    const int lim = max_lds_per_block();
    const int cus = std::max(1, cu_count());
    int waves = 1;
    while (waves < 16 && (int64_t)waves * cus < chains) waves <<= 1;
    while (waves > 1 && soa + per * waves > (size_t)lim) waves >>= 1;
    if (soa + per * waves <= (size_t)lim && (waves >= 4 || (int64_t)waves * cus >= chains)) {
      sa::StaticParams sp{(uint32_t)model->d0, (uint32_t)model->d2,
                          (1ull << 32) / (uint64_t)model->max_batch + 1};
      const size_t lds = soa + per * waves;
      const sa::QueuePtrs qp = dev_queue(queue);
      const uint64_t st = model->swap_threshold;
      hipError_t e = hipSuccess;
      switch (lg) {
        case 0: e = launch_static<0, OBJ>(waves, lds, dm, sp, qp, chains, iters, T0, alpha, seed, st, srch, w, stream); break;
        case 1: e = launch_static<1, OBJ>(waves, lds, dm, sp, qp, chains, iters, T0, alpha, seed, st, srch, w, stream); break;
        case 2: e = launch_static<2, OBJ>(waves, lds, dm, sp, qp, chains, iters, T0, alpha, seed, st, srch, w, stream); break;
        case 3: e = launch_static<3, OBJ>(waves, lds, dm, sp, qp, chains, iters, T0, alpha, seed, st, srch, w, stream); break;
        case 4: e = launch_static<4, OBJ>(waves, lds, dm, sp, qp, chains, iters, T0, alpha, seed, st, srch, w, stream); break;
        case 5: e = launch_static<5, OBJ>(waves, lds, dm, sp, qp, chains, iters, T0, alpha, seed, st, srch, w, stream); break;
        default: {
          if (lds > 65536) {
            e = hipFuncSetAttribute(reinterpret_cast<const void *>(&sa::anneal_wave_kernel<OBJ>),
                                    hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
            if (e != hipSuccess) break;
          }
          const int grid = (chains + waves - 1) / waves;
          sa::anneal_wave_kernel<OBJ><<<grid, waves * 64, lds, stream>>>(dm, sp, qp, chains, iters, T0, alpha,
                                                                         (uint32_t)seed, (uint32_t)(seed >> 32), st,
                                                                         srch, w);
          e = hipGetLastError();
          break;
        }
      }
      if (e != hipSuccess) return hip_fail(e);
      done = true;
    }
  }
  if (!done && model->policy == SCHED_CONTINUOUS && (dm.flags & sa::kFlagNarrowPrefill)) {
    const bool ls = (dm.flags & sa::kFlagListSched) != 0;
    const size_t soa = (size_t)n * 16;
    const bool inc = ls && std::min(model->max_batch, n) <= 32;
    const size_t per = (((size_t)n * 2 + 15) & ~size_t(15)) + (ls ? ((sa::cont_ls_scratch_bytes(n) + 15) & ~size_t(15)) : 0) +
                       (inc ? sa::cont_inc_bytes(n, model->max_batch) : 0);
    const int cus = std::max(1, cu_count());
    const int lim = max_lds_per_block();
    int waves = 1;
    while (waves < 16 && (int64_t)waves * cus < chains) waves <<= 1;
    while (waves > 1 && soa + per * waves > (size_t)lim) waves >>= 1;
    const size_t lds = soa + per * waves;
    if (lds <= (size_t)lim) {
      const void *fn =
          ls ? (const void *)&sa::anneal_cont_kernel<true, OBJ> : (const void *)&sa::anneal_cont_kernel<false, OBJ>;
      if (lds > 65536) HIP_TRY(hipFuncSetAttribute(fn, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds));
      const int grid = (chains + waves - 1) / waves;
      if (ls) {
        sa::anneal_cont_kernel<true, OBJ><<<grid, waves * 64, lds, stream>>>(
            dm, dev_queue(queue), chains, iters, T0, alpha, (uint32_t)seed, (uint32_t)(seed >> 32), model->swap_threshold,
            srch, w);
      } else {
        sa::anneal_cont_kernel<false, OBJ><<<grid, waves * 64, lds, stream>>>(
            dm, dev_queue(queue), chains, iters, T0, alpha, (uint32_t)seed, (uint32_t)(seed >> 32), model->swap_threshold,
            srch, w);
      }
      HIP_TRY(hipGetLastError());
      done = true;
    }
  }
  if (!done) {
    const int grid = (chains + sa::kWavesPerBlock - 1) / sa::kWavesPerBlock;
    sa::anneal_kernel<OBJ><<<grid, sa::kBlock, anneal_lds_bytes(n), stream>>>(
        dm, dev_queue(queue), chains, iters, T0, alpha, (uint32_t)seed, (uint32_t)(seed >> 32), model->swap_threshold,
        srch, w);
    HIP_TRY(hipGetLastError());
  }
  return SCHED_OK;
}

template <int LG, int OBJ>
hipError_t launch_multi_static_lg(int grid, int waves, size_t lds, const sa::DevModel &dm, const sa::StaticParams &sp,
                                  int n, int instances, int chains, int groups, int iters, double T0, double alpha,
                                  uint64_t seed, uint64_t swap_thr, const sa::SearchParams &srch, unsigned char *w,
                                  hipStream_t stream) {
  if (lds > 65536) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void *>(&sa::multi_static_kernel<LG, OBJ>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  sa::multi_static_kernel<LG, OBJ><<<grid, waves * 64, lds, stream>>>(dm, sp, n, instances, chains, groups, iters, T0,
                                                                      alpha, (uint32_t)seed, (uint32_t)(seed >> 32),
                                                                      swap_thr, srch, w);
  return hipGetLastError();
}

// Every instance's chains on the static delta kernels, with as many chains per workgroup as
// the single-queue launch would take for all of them (LDS for the largest instance); sets
// `done` when the LDS allows it.
template <int OBJ>
int launch_multi_static(const sched_model_t *model, const sa::DevModel &dm, int n, int nk_max, int instances,
                        int chains, int total, int iters, double T0, double alpha, uint64_t seed,
                        const sa::SearchParams &srch, unsigned char *w, hipStream_t stream, bool &done) {
  int lg = 0;
  while ((1 << lg) < model->max_batch) ++lg;
  const size_t soa = (size_t)(nk_max + 1) * 16;
  const size_t per = lg == 6 ? wave_chain_lds(nk_max, model->max_batch) : static_wave_lds(nk_max, model->max_batch);
  const int lim = max_lds_per_block(), cus = std::max(1, cu_count());
  int waves = 1;
  while (waves < 16 && waves < chains && (int64_t)waves * cus < total) waves <<= 1;
  while (waves > 1 && soa + per * waves > (size_t)lim) waves >>= 1;
  if (soa + per * waves > (size_t)lim || (waves < 4 && (int64_t)waves * cus < total)) return SCHED_OK;
  const sa::StaticParams sp{(uint32_t)model->d0, (uint32_t)model->d2, (1ull << 32) / (uint64_t)model->max_batch + 1};
  const size_t lds = soa + per * waves;
  const int groups = (chains + waves - 1) / waves, grid = instances * groups;
  const uint64_t st = model->swap_threshold;
  hipError_t e = hipSuccess;
  switch (lg) {
#define SA_MULTI_LG(L)                                                                                            \
  case L:                                                                                                          \
    e = launch_multi_static_lg<L, OBJ>(grid, waves, lds, dm, sp, n, instances, chains, groups, iters, T0, alpha, \
                                       seed, st, srch, w, stream);                                               \
    break;
    SA_MULTI_LG(0)
    SA_MULTI_LG(1)
    SA_MULTI_LG(2)
    SA_MULTI_LG(3)
    SA_MULTI_LG(4)
    SA_MULTI_LG(5)
    SA_MULTI_LG(6)
#undef SA_MULTI_LG
    default: return SCHED_EINVAL;
  }
  if (e != hipSuccess) return hip_fail(e);
  done = true;
  return SCHED_OK;
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
  if (!queue || queue->n < 1 || queue->n > SCHED_MAX_N) return SCHED_EINVAL;
  int rc = check_model(model, queue->n);
  if (rc) return rc;
  if (k > 0 && (!perms || !out)) return SCHED_EINVAL;
  HostQueue h;
  if ((rc = fetch_queue(queue, stream, h))) return rc;
  if ((rc = range_check(h, model, queue->n))) return rc;
  if (k == 0) return SCHED_OK;
  const int n = queue->n;
  const sa::DevModel dm = dev_model(model, n, prefill_narrow(h, model, n), list_sched_ok(h, model, n),
                                    timeline_narrow(h, model, n));
  if (model->policy != SCHED_CONTINUOUS && static_narrow(h, model, n)) {
    int lg = 0;
    while ((1 << lg) < model->max_batch) ++lg;
    const sa::StaticParams sp{(uint32_t)model->d0, (uint32_t)model->d2, (1ull << 32) / (uint64_t)model->max_batch + 1};
    const size_t lds = (size_t)(n + 1) * 16 + ((((size_t)n * 2 + 15) & ~size_t(15)) + 64 * 8 + 32 * 4) * 4;
    const int64_t want4 = (k + 3) / 4;
    const int g4 = (int)std::min<int64_t>(want4, 256 * 32);
    const bool t32 = sized_narrow(h, model, n);  // the whole timeline in 32 bits
    hipError_t e = hipSuccess;
#define SA_EVAL_CASE(L)                                                                                            \
  case L:                                                                                                        \
    if (detail)                                                                                                  \
      sa::eval_static_kernel<L, true><<<g4, 256, lds, stream>>>(dm, sp, dev_queue(queue), perms, k, out, detail);  \
    else if (t32)                                                                                                \
      sa::eval_static_kernel<L, false, true><<<g4, 256, lds, stream>>>(dm, sp, dev_queue(queue), perms, k, out,     \
                                                                       nullptr);                                 \
    else                                                                                                         \
      sa::eval_static_kernel<L, false><<<g4, 256, lds, stream>>>(dm, sp, dev_queue(queue), perms, k, out, nullptr); \
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
    e = hipGetLastError();
    if (e != hipSuccess) return hip_fail(e);
    return SCHED_OK;
  }
  // one order per wave, up to four waves per workgroup as the LDS allows
  const bool ls = dm.policy == SCHED_CONTINUOUS && (dm.flags & sa::kFlagListSched);
  int waves = sa::kWavesPerBlock;
  while (waves > 1 && eval_lds_bytes(n, ls, waves) > (size_t)max_lds_per_block()) waves >>= 1;
  const size_t lds = eval_lds_bytes(n, ls, waves);
  const int grid = (int)std::min<int64_t>((k + waves - 1) / waves, 256 * 32);
  if (lds > 65536) {
    HIP_TRY(hipFuncSetAttribute(reinterpret_cast<const void *>(detail ? (const void *)&sa::eval_kernel<true>
                                                                      : (const void *)&sa::eval_kernel<false>),
                                hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds));
  }
  if (detail) {
    sa::eval_kernel<true><<<grid, waves * 64, lds, stream>>>(dm, dev_queue(queue), perms, k, out, detail);
  } else {
    sa::eval_kernel<false><<<grid, waves * 64, lds, stream>>>(dm, dev_queue(queue), perms, k, out, nullptr);
  }
  HIP_TRY(hipGetLastError());
  return SCHED_OK;
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
  if (!queue || queue->n < 1 || queue->n > SCHED_MAX_N) return SCHED_EINVAL;
  if (chains < 1 || iters < 0 || !(T0 > 0.0) || !std::isfinite(T0) || !(alpha > 0.0) || !std::isfinite(alpha))
    return SCHED_EINVAL;
  sa::SearchParams srch{SCHED_OBJ_LEX, 1, 0, 0};
  if (search) {
    if ((search->objective != SCHED_OBJ_LEX && search->objective != SCHED_OBJ_RATIO) || search->level_len < 1 ||
        (search->early_exit != 0 && search->early_exit != 1) || search->reserved != 0)
      return SCHED_EINVAL;
    srch = sa::SearchParams{search->objective, search->level_len, search->early_exit, 0};
  }
  int rc = check_model(model, queue->n);
  if (rc) return rc;
  // the ratio needs a positive total latency: every request takes at least p0 + d0 + d1
  if (srch.objective == SCHED_OBJ_RATIO && model->p0 + model->d0 + model->d1 < 1) return SCHED_EINVAL;
  if (!ws || (reinterpret_cast<uintptr_t>(ws) & 255u)) return SCHED_EINVAL;
  if (ws_bytes < sched_ws_bytes(queue->n, chains)) return SCHED_ENOSPC;
  HostQueue h;
  if ((rc = fetch_queue(queue, stream, h))) return rc;
  if ((rc = range_check(h, model, queue->n))) return rc;
  if (srch.objective == SCHED_OBJ_RATIO && (rc = ratio_range_check(h, model, queue->n))) return rc;
  const int n = queue->n;
  const sa::DevModel dm = dev_model(model, n, prefill_narrow(h, model, n), list_sched_ok(h, model, n),
                                    timeline_narrow(h, model, n), timeline_bound(h, model, n) < std::ldexp(1.0L, 57));
  unsigned char *w = static_cast<unsigned char *>(ws);
  sa::start_kernel<<<1, 1024, 0, stream>>>(dm, dev_queue(queue), chains, iters, model->t_ref_us, srch, w);
  HIP_TRY(hipGetLastError());
  rc = srch.objective ? launch_chains<1>(h, model, dm, queue, chains, iters, T0, alpha, seed, srch, w, stream)
                      : launch_chains<0>(h, model, dm, queue, chains, iters, T0, alpha, seed, srch, w, stream);
  if (rc) return rc;
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
  if (!queue || queue->n < 1 || queue->n > SCHED_MAX_N) return SCHED_EINVAL;
  int rc = check_model(model, queue->n);
  if (rc) return rc;
  if (model->policy == SCHED_CONTINUOUS) return SCHED_EINVAL;
  if (k > 0 && (!perms || !starts || !out)) return SCHED_EINVAL;
  HostQueue h;
  if ((rc = fetch_queue(queue, stream, h))) return rc;
  if ((rc = range_check(h, model, queue->n))) return rc;
  if (k == 0) return SCHED_OK;
  const int n = queue->n;
  sa::DevModel dm = dev_model(model, n, false, false, false, timeline_bound(h, model, n) < std::ldexp(1.0L, 57),
                              static_narrow(h, model, n));
  if (sized_narrow(h, model, n)) dm.flags |= sa::kFlagTime32;  // every layout's timeline in 32 bits
  const size_t pb = ((size_t)n * 2 + 15) & ~size_t(15), fb = ((size_t)n + 15) & ~size_t(15);
  const size_t lds = (((size_t)n * 16 + 15) & ~size_t(15)) + 4 * (pb + fb + 64 * 16 + 32 * 4);
  const int grid = (int)std::min<int64_t>((k + 3) / 4, 256 * 32);
  if (detail)
    sa::eval_sized_kernel<true><<<grid, 256, lds, stream>>>(dm, dev_queue(queue), perms, starts, k, out, detail);
  else
    sa::eval_sized_kernel<false><<<grid, 256, lds, stream>>>(dm, dev_queue(queue), perms, starts, k, out, nullptr);
  HIP_TRY(hipGetLastError());
  return SCHED_OK;
}

int sched_starts(const void *ws, uint8_t *cur_starts, uint8_t *best_starts, uint8_t *winner_starts,
                 hipStream_t stream) {
  if (!ws || (!cur_starts && !best_starts && !winner_starts)) return SCHED_EINVAL;
  sa::starts_copy_kernel<<<256, 256, 0, stream>>>(static_cast<const unsigned char *>(ws), cur_starts, best_starts,
                                                  winner_starts);
  HIP_TRY(hipGetLastError());
  return SCHED_OK;
}

int sched_assign(const sched_queue_t *queue, int32_t instances, const int64_t *capacity, int32_t *inst_out,
                 hipStream_t stream) {
  if (!queue || queue->n < 1 || queue->n > SCHED_MAX_N) return SCHED_EINVAL;
  if (instances < 1 || instances > SCHED_MAX_INSTANCES || !capacity || !inst_out) return SCHED_EINVAL;
  HostQueue h;
  int rc = fetch_queue(queue, stream, h);
  if (rc) return rc;
  std::vector<int64_t> cap((size_t)instances);
  HIP_TRY(hipMemcpyAsync(cap.data(), capacity, (size_t)instances * 8, hipMemcpyDeviceToHost, stream));
  HIP_TRY(hipStreamSynchronize(stream));
  bool narrow = true;
  for (int64_t c : cap) {
    if (c < 1 || c > (int64_t(1) << 48)) return SCHED_EINVAL;
    narrow = narrow && c < sa::kAssignNarrowCap;
  }
  if (narrow)
    sa::assign_sorted_kernel<<<1, 64, 0, stream>>>(dev_queue(queue), queue->n, instances, capacity, inst_out);
  else
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
  if (!queue || queue->n < 1 || queue->n > SCHED_MAX_N) return SCHED_EINVAL;
  if (instances < 1 || instances > SCHED_MAX_INSTANCES || !inst_of) return SCHED_EINVAL;
  if (chains < 1 || iters < 0 || !(T0 > 0.0) || !std::isfinite(T0) || !(alpha > 0.0) || !std::isfinite(alpha))
    return SCHED_EINVAL;
  sa::SearchParams srch{SCHED_OBJ_LEX, 1, 0, 0};
  if (search) {
    if ((search->objective != SCHED_OBJ_LEX && search->objective != SCHED_OBJ_RATIO) || search->level_len < 1 ||
        (search->early_exit != 0 && search->early_exit != 1) || search->reserved != 0)
      return SCHED_EINVAL;
    srch = sa::SearchParams{search->objective, search->level_len, search->early_exit, 0};
  }
  int rc = check_model(model, queue->n);
  if (rc) return rc;
  if (model->policy == SCHED_STATIC_SEARCH) return SCHED_EINVAL;
  if (srch.objective == SCHED_OBJ_RATIO && model->p0 + model->d0 + model->d1 < 1) return SCHED_EINVAL;
  const int n = queue->n;
  if (!ws || (reinterpret_cast<uintptr_t>(ws) & 255u)) return SCHED_EINVAL;
  if (ws_bytes < sched_ws_bytes_multi(n, instances, chains)) return SCHED_ENOSPC;
  HostQueue h;
  if ((rc = fetch_queue(queue, stream, h))) return rc;
  std::vector<int32_t> inst((size_t)n);
  HIP_TRY(hipMemcpyAsync(inst.data(), inst_of, (size_t)n * 4, hipMemcpyDeviceToHost, stream));
  HIP_TRY(hipStreamSynchronize(stream));
  std::vector<int> cnt((size_t)instances, 0);
  for (int32_t v : inst) {
    if (v < 0 || v >= instances) return SCHED_EINVAL;
    ++cnt[(size_t)v];
  }
  // every instance's queue is part of the whole one, so the whole queue's bounds hold for it
  if ((rc = range_check(h, model, n))) return rc;
  if (srch.objective == SCHED_OBJ_RATIO && (rc = ratio_range_check(h, model, n))) return rc;
  const int nk_max = *std::max_element(cnt.begin(), cnt.end());
  const sa::DevModel dm = dev_model(model, n, prefill_narrow(h, model, n), list_sched_ok(h, model, n),
                                    timeline_narrow(h, model, n));
  unsigned char *w = static_cast<unsigned char *>(ws);
  sa::multi_header_kernel<<<1, 1, 0, stream>>>(w, n, instances, chains, (int64_t)sa::mws_slot_bytes(n, chains));
  HIP_TRY(hipGetLastError());
  sa::gather_kernel<<<instances, 1024, 0, stream>>>(dev_queue(queue), n, inst_of, chains, instances, w);
  HIP_TRY(hipGetLastError());
  sa::multi_start_kernel<<<instances, 1024, 0, stream>>>(dm, n, instances, chains, iters, model->t_ref_us, srch, w);
  HIP_TRY(hipGetLastError());
  bool done = nk_max == 0;
  if (!done && model->policy == SCHED_STATIC &&
      sa::reg_parts(nk_max, model->max_batch) > 0 &&
      static_narrow(h, model, n)) {
    // every instance small: the register kernel per instance, no LDS (two or three positions
    // per lane when an instance holds more than 64 requests)
    const bool two = nk_max > 64;
    const int total = instances * chains, cus = std::max(1, cu_count());
    const int waves = total >= 4 * cus && chains >= 4 ? 4 : (total >= 2 * cus && chains >= 2 ? 2 : 1);
    const int groups = (chains + waves - 1) / waves, grid = instances * groups;
    const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
    const uint64_t st = model->swap_threshold;
    // every instance's timeline is within the whole queue's bound
    sa::DevModel dr = dm;
    if (sized_narrow(h, model, n)) dr.flags |= sa::kFlagTime32;
#define SA_MULTI_REG(LG)                                                                                         \
  if (two && srch.objective)                                                                                   \
    sa::multi_reg_h_kernel<LG, 1><<<grid, waves * 64, 0, stream>>>(dr, n, instances, chains, groups, iters, T0,    \
                                                                  alpha, k0, k1, st, srch, w);                 \
  else if (two)                                                                                                \
    sa::multi_reg_h_kernel<LG, 0><<<grid, waves * 64, 0, stream>>>(dr, n, instances, chains, groups, iters, T0,    \
                                                                  alpha, k0, k1, st, srch, w);                 \
  else if (srch.objective)                                                                                     \
    sa::multi_reg_kernel<LG, 1><<<grid, waves * 64, 0, stream>>>(dr, n, instances, chains, groups, iters, T0,     \
                                                                 alpha, k0, k1, st, srch, w);                  \
  else                                                                                                         \
    sa::multi_reg_kernel<LG, 0><<<grid, waves * 64, 0, stream>>>(dr, n, instances, chains, groups, iters, T0,     \
                                                                 alpha, k0, k1, st, srch, w);
    switch (model->max_batch) {
      case 1: SA_MULTI_REG(0) break;
      case 2: SA_MULTI_REG(1) break;
      case 4: SA_MULTI_REG(2) break;
      case 8: SA_MULTI_REG(3) break;
      default: SA_MULTI_REG(4) break;
    }
#undef SA_MULTI_REG
    HIP_TRY(hipGetLastError());
    done = true;
  }
  if (!done && model->policy == SCHED_STATIC && static_narrow(h, model, n)) {
    // every instance's queue is part of the whole one, so the delta kernel's widths hold
    const int total = instances * chains;
    if (srch.objective)
      rc = launch_multi_static<1>(model, dm, n, nk_max, instances, chains, total, iters, T0, alpha, seed, srch, w,
                                  stream, done);
    else
      rc = launch_multi_static<0>(model, dm, n, nk_max, instances, chains, total, iters, T0, alpha, seed, srch, w,
                                  stream, done);
    if (rc) return rc;
  }
  if (!done) {
    const int groups = (chains + sa::kWavesPerBlock - 1) / sa::kWavesPerBlock;
    const size_t lds = anneal_lds_bytes(nk_max);
    const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
    if (srch.objective)
      sa::multi_anneal_kernel<1><<<instances * groups, sa::kBlock, lds, stream>>>(
          dm, n, instances, chains, groups, iters, T0, alpha, k0, k1, model->swap_threshold, srch, w);
    else
      sa::multi_anneal_kernel<0><<<instances * groups, sa::kBlock, lds, stream>>>(
          dm, n, instances, chains, groups, iters, T0, alpha, k0, k1, model->swap_threshold, srch, w);
    HIP_TRY(hipGetLastError());
  }
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
  if (!queue || queue->n < 1 || queue->n > SCHED_MAX_N) return SCHED_EINVAL;
  int rc = check_fit(fit);
  if (rc) return rc;
  if (k > 0 && (!perms || !out)) return SCHED_EINVAL;
  HostQueue h;
  if ((rc = fetch_queue(queue, stream, h, tpot_thr ? 3 : 2))) return rc;
  if ((rc = fit_range_check(h, fit, queue->n, false))) return rc;
  if (k == 0) return SCHED_OK;
  const int n = queue->n;
  const size_t pb = ((size_t)n * 2 + 15) & ~size_t(15), fb = ((size_t)n + 15) & ~size_t(15);
  const size_t lds = (((size_t)n * 16 + 15) & ~size_t(15)) + 4 * (pb + fb + 32 * 4);
  const int grid = (int)std::min<int64_t>((k + 3) / 4, 256 * 32);
  const sa::DevFit df = dev_fit(fit, n, fit_timeline_bound(h, fit, n) < std::ldexp(1.0L, 57));
  if (detail)
    sa::eval_fit_kernel<true><<<grid, 256, lds, stream>>>(df, dev_queue(queue), tpot_thr, perms, starts, k, out, detail);
  else
    sa::eval_fit_kernel<false><<<grid, 256, lds, stream>>>(df, dev_queue(queue), tpot_thr, perms, starts, k, out,
                                                           nullptr);
  HIP_TRY(hipGetLastError());
  return SCHED_OK;
}

int sched_anneal_fit(const sched_queue_t *queue, const sched_fit_model_t *fit, const uint32_t *tpot_thr,
                     const sched_search_t *search, int32_t chains, int32_t iters, double T0, double alpha,
                     uint64_t seed, void *ws, size_t ws_bytes, hipStream_t stream) {
  if (!queue || queue->n < 1 || queue->n > SCHED_MAX_N) return SCHED_EINVAL;
  if (chains < 1 || iters < 0 || !(T0 > 0.0) || !std::isfinite(T0) || !(alpha > 0.0) || !std::isfinite(alpha))
    return SCHED_EINVAL;
  sa::SearchParams srch{SCHED_OBJ_LEX, 1, 0, 0};
  if (search) {
    if ((search->objective != SCHED_OBJ_LEX && search->objective != SCHED_OBJ_RATIO) || search->level_len < 1 ||
        (search->early_exit != 0 && search->early_exit != 1) || search->reserved != 0)
      return SCHED_EINVAL;
    srch = sa::SearchParams{search->objective, search->level_len, search->early_exit, 0};
  }
  int rc = check_fit(fit);
  if (rc) return rc;
  if (srch.objective == SCHED_OBJ_RATIO && fit->dp + fit->dd < 1) return SCHED_EINVAL;  // positive latencies
  if (!ws || (reinterpret_cast<uintptr_t>(ws) & 255u)) return SCHED_EINVAL;
  if (ws_bytes < sched_ws_bytes(queue->n, chains)) return SCHED_ENOSPC;
  HostQueue h;
  if ((rc = fetch_queue(queue, stream, h, tpot_thr ? 3 : 2))) return rc;
  if ((rc = fit_range_check(h, fit, queue->n, srch.objective == SCHED_OBJ_RATIO))) return rc;
  const int n = queue->n;
  const sa::DevFit df = dev_fit(fit, n, fit_timeline_bound(h, fit, n) < std::ldexp(1.0L, 57),
                                fit_member_bound(h, fit, n) < 4294967295.0L);
  unsigned char *w = static_cast<unsigned char *>(ws);
  sa::start_fit_kernel<<<1, 1024, 0, stream>>>(df, dev_queue(queue), tpot_thr, chains, iters, fit->t_ref, srch, w);
  HIP_TRY(hipGetLastError());
  const uint32_t k0 = (uint32_t)seed, k1 = (uint32_t)(seed >> 32);
  if (n <= 64 && df.win) {
    // small queue: order, request fields and layout in registers, no LDS
    const int cus = std::max(1, cu_count());
    const int waves = chains >= 4 * cus ? 4 : (chains >= 2 * cus ? 2 : 1);
    const int rgrid = (chains + waves - 1) / waves;
    if (srch.objective)
      sa::anneal_reg_fit_kernel<1><<<rgrid, waves * 64, 0, stream>>>(df, dev_queue(queue), tpot_thr, chains, iters, T0,
                                                                     alpha, k0, k1, fit->swap_threshold, srch, w);
    else
      sa::anneal_reg_fit_kernel<0><<<rgrid, waves * 64, 0, stream>>>(df, dev_queue(queue), tpot_thr, chains, iters, T0,
                                                                     alpha, k0, k1, fit->swap_threshold, srch, w);
    HIP_TRY(hipGetLastError());
  } else {
    const size_t pb = ((size_t)n * 2 + 15) & ~size_t(15), fb = ((size_t)n + 15) & ~size_t(15);
    const size_t lds = (((size_t)n * 16 + 15) & ~size_t(15)) + 4 * (2 * pb + 2 * fb);
    const int grid = (chains + 3) / 4;
    if (srch.objective)
      sa::anneal_fit_kernel<1><<<grid, 256, lds, stream>>>(df, dev_queue(queue), tpot_thr, chains, iters, T0, alpha, k0,
                                                           k1, fit->swap_threshold, srch, w);
    else
      sa::anneal_fit_kernel<0><<<grid, 256, lds, stream>>>(df, dev_queue(queue), tpot_thr, chains, iters, T0, alpha, k0,
                                                           k1, fit->swap_threshold, srch, w);
    HIP_TRY(hipGetLastError());
  }
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
