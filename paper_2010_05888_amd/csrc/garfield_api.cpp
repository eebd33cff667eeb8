// C-ABI of libgarfield: argument validation (the requirements of Section 3.1
// of the paper), the per-device workspace, and the launch sequence of each
// aggregation rule on the caller's stream. See include/garfield.h.

#include <hip/hip_runtime.h>

#include <cmath>
#include <map>
#include <mutex>
#include <new>
#include <vector>

#include "garfield.h"
#include "garfield_tuning.h"
#include "dist_layout.h"
#include "internal.h"
#include "timing.h"

// Scratch of garfield_multikrum_noalloc: a fixed array in every device's
// memory, held from the library's load until the process ends. Host code
// never uses the name itself (on the host it is only a stand-in for the
// symbol): the device address comes from hipGetSymbolAddress, once per
// device (static_scratch below), and every kernel argument and carve uses
// that address.
static __device__ __align__(256) unsigned char scratch[GARFIELD_NOALLOC_SCRATCH_BYTES];

namespace garfield {
namespace {

struct DeviceWorkspace {
  void* ptr = nullptr;
  size_t bytes = 0;
};

std::mutex g_mutex;
std::map<int, DeviceWorkspace> g_workspaces;

garfield_status to_status(hipError_t e) {
  if (e == hipSuccess) return GARFIELD_OK;
  (void)hipGetLastError();  // clear the sticky launch error for the next call
  return GARFIELD_EHIP;
}

// Workspace of the current device with at least `need` bytes. Growing it
// waits for the device to go idle before the old buffer is freed.
garfield_status workspace(size_t need, void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return to_status(hipErrorInvalidDevice);
  std::lock_guard<std::mutex> lock(g_mutex);
  DeviceWorkspace& w = g_workspaces[dev];
  if (w.bytes < need) {
    if (w.ptr) {
      if (hipDeviceSynchronize() != hipSuccess) return to_status(hipErrorUnknown);
      (void)hipFree(w.ptr);
      w.ptr = nullptr;
      w.bytes = 0;
    }
    size_t alloc = need < (size_t{1} << 20) ? (size_t{1} << 20) : need;
    alloc = (alloc + 0xFFFFF) & ~size_t{0xFFFFF};
    if (hipMalloc(&w.ptr, alloc) != hipSuccess) {
      (void)hipGetLastError();
      w.ptr = nullptr;
      return GARFIELD_ENOMEM;
    }
    w.bytes = alloc;
  }
  *out = w.ptr;
  return GARFIELD_OK;
}

size_t align256(size_t b) { return (b + 255) & ~size_t{255}; }

// Checks shared by every rule.
garfield_status check_common(const float* x, int n, int f, int64_t d) {
  if (n < 1 || f < 0 || d < 0) return GARFIELD_EINVAL;
  if (d > 0 && (!x || reinterpret_cast<uintptr_t>(x) % sizeof(float) != 0)) return GARFIELD_EINVAL;
  if (n > GARFIELD_NMAX) return GARFIELD_ETOOBIG;
  // every kernel covers d in one launch of at most 2^31 - 1 workgroups of
  // kBlock lanes, each lane at least one coordinate
  if (d > int64_t{0x7fffffff} * kBlock) return GARFIELD_ETOOBIG;
  return GARFIELD_OK;
}

// Distance step into the workspace. *ds receives the entry sums (valid once
// the stream reaches the end of the step). `extra` bytes of scratch follow
// the distance workspace and are returned in *extra_ptr.
// fold_entries > 0: the consumer is a selection kernel of fold_entries / 4
// waves that reads D through load_dist, so a direct-engine step with few
// tiles and at most fold_entries entries skips the tile-sum kernel (the
// selection kernel adds the tiles in the same order).
constexpr int kFoldSelect = 4 * 16;  // k_krum_select, k_bulyan_select, k_mda_cover: 16 waves
constexpr int kFoldMda = 4 * 4;      // k_mda_search: 4 waves
// colsum: the scratch begins with d doubles that receive the column sums
// (enqueue_distances' colsum).
// The steps of run_distances on scratch the caller provides (`base`, at least
// dist_workspace_bytes(plan) + align256(extra) bytes).
garfield_status run_distances_on(const DistPlan& plan, void* base, const float* x, size_t extra,
                                 DistSums* ds, void** extra_ptr, hipStream_t s,
                                 int fold_entries, bool colsum);

garfield_status run_distances(const float* x, int n, int64_t d, size_t extra, DistSums* ds,
                              void** extra_ptr, hipStream_t s, int fold_entries = 0,
                              bool colsum = false) {
  const DistPlan plan = plan_distances(n, d, x);
  const size_t dist_bytes = dist_workspace_bytes(plan);
  void* base = nullptr;
  garfield_status st = workspace(dist_bytes + align256(extra), &base);
  if (st != GARFIELD_OK) return st;
  return run_distances_on(plan, base, x, extra, ds, extra_ptr, s, fold_entries, colsum);
}

garfield_status run_distances_on(const DistPlan& plan, void* base, const float* x, size_t extra,
                                 DistSums* ds, void** extra_ptr, hipStream_t s,
                                 int fold_entries, bool colsum) {
  (void)extra;
  const size_t dist_bytes = dist_workspace_bytes(plan);
  const DistWorkspace ws = carve_dist_workspace(plan, base);
  *ds = dist_sums(plan, ws);
  if (extra_ptr) *extra_ptr = static_cast<char*>(base) + dist_bytes;
  const bool fold = fold_entries > 0 && foldable(plan, fold_entries);
  if (fold) {
    ds->partial = ws.partial;
    ds->tiles = plan.tiles;
  }
  double* cs = colsum ? static_cast<double*>(*extra_ptr) : nullptr;
  return to_status(enqueue_distances(x, plan, ws, s, !fold, cs));
}

// The mean of m of the n rows reads m rows. With the column sums of the
// distance step (d doubles written there, read here) it reads those and the
// n - m other rows instead: fewer bytes when 2m > n + 4. Direct engine with
// n <= kColSumMaxN only.
bool use_colsum(const float* x, int n, int64_t d, int m) {
  if (d == 0 || n > kColSumMaxN || 2 * m <= n + 4) return false;
  return plan_distances(n, d, x).engine == kEngineDirect;
}
size_t colsum_bytes(bool cs, int64_t d) {
  return cs ? static_cast<size_t>(d) * sizeof(double) : 0;
}

// Requirements of `rule` (Section 3.1) and the number of indices it selects
// (0: no selection). m <= 0 means n - f for Multi-Krum.
garfield_status rule_shape(int rule, int n, int f, int* m, int* k) {
  if (n < 1 || f < 0) return GARFIELD_EINVAL;
  if (n > GARFIELD_NMAX) return GARFIELD_ETOOBIG;
  switch (rule) {
    case GARFIELD_RULE_KRUM:
    case GARFIELD_RULE_MULTIKRUM:
    case GARFIELD_RULE_MULTIKRUM_ITERATED:
      if (n < 2 * f + 3) return GARFIELD_EREQ;
      if (rule == GARFIELD_RULE_KRUM) *m = 1;
      if (*m <= 0) *m = n - f;
      if (*m > n - f) return GARFIELD_EINVAL;
      *k = *m;
      return GARFIELD_OK;
    case GARFIELD_RULE_BULYAN:
      if (n < 4 * f + 3) return GARFIELD_EREQ;
      *k = n - 2 * f;
      return GARFIELD_OK;
    case GARFIELD_RULE_MDA: {
      if (n < 2 * f + 1) return GARFIELD_EREQ;
      const int64_t subsets = binomial(n, f);
      if (subsets < 0 || subsets > GARFIELD_MDA_MAX_SUBSETS) return GARFIELD_ETOOBIG;
      *k = n - f;
      return GARFIELD_OK;
    }
    case GARFIELD_RULE_MEDIAN:
      if (n < 2 * f + 1) return GARFIELD_EREQ;
      *k = 0;
      return GARFIELD_OK;
    case GARFIELD_RULE_AVERAGE:
      *k = 0;
      return GARFIELD_OK;
    default:
      return GARFIELD_EINVAL;
  }
}

std::mutex g_scratch_mutex;
std::map<int, void*> g_scratch_ptr;  // device -> address of `scratch` there

garfield_status static_scratch(void** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return to_status(hipErrorInvalidDevice);
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  auto it = g_scratch_ptr.find(dev);
  if (it == g_scratch_ptr.end()) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) return to_status(e != hipSuccess ? e : hipErrorUnknown);
    it = g_scratch_ptr.emplace(dev, p).first;
  }
  *out = it->second;
  return GARFIELD_OK;
}

static_assert(GARFIELD_NMAX == kNmax, "kernel limit and public limit differ");
static_assert(GARFIELD_DIRECT_MAX_N_LIMIT == kDirectMaxNLimit, "direct engine limit differs");

}  // namespace
}  // namespace garfield

using namespace garfield;

// A segmented aggregation: the running sum of the segments' distance matrices
// and the selection made from it, on the device that created it.
struct garfield_segmented {
  int rule = 0, n = 0, f = 0, m = 0, k = 0;
  int device = 0;
  double* dacc = nullptr;   // n x n fp64
  int32_t* sel = nullptr;   // n int32 (the first k hold the selection)
  bool selected = false;    // a selection has been enqueued since the last reset
};

extern "C" {

garfield_status garfield_pairwise_sqdist(const float* x, int n, int64_t d, double* dist,
                                         void* stream) {
  garfield_status st = check_common(x, n, 0, d);
  if (st != GARFIELD_OK) return st;
  if (!dist) return GARFIELD_EINVAL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  DistSums ds;
  st = run_distances(x, n, d, 0, &ds, nullptr, s);
  if (st != GARFIELD_OK) return st;
  return to_status(enqueue_write_dist(ds, dist, s));
}

garfield_status garfield_multikrum(const float* x, int n, int f, int64_t d, int m, float* out,
                                   int32_t* sel, void* stream) {
  garfield_status st = check_common(x, n, f, d);
  if (st != GARFIELD_OK) return st;
  if (!sel) return GARFIELD_EINVAL;
  if (n < 2 * f + 3) return GARFIELD_EREQ;
  if (m <= 0) m = n - f;
  if (m > n - f) return GARFIELD_EINVAL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  DistSums ds;
  const DistPlan plan = plan_distances(n, d, x);
  if (krum_fusable(plan, out)) {  // short input: selection and mean in one kernel
    st = run_distances(x, n, d, 0, &ds, nullptr, s, plan.entries);
    if (st != GARFIELD_OK) return st;
    return to_status(enqueue_krum_select_mean(x, ds, d, f, m, sel, out, s));
  }
  const bool cs = out && use_colsum(x, n, d, m);
  void* colsum = nullptr;
  st = run_distances(x, n, d, colsum_bytes(cs, d), &ds, &colsum, s, kFoldSelect, cs);
  if (st != GARFIELD_OK) return st;
  st = to_status(enqueue_krum_select(ds, f, m, sel, s));
  if (st != GARFIELD_OK || !out) return st;
  if (cs)
    return to_status(enqueue_mean_complement(x, n, d, sel, m, static_cast<double*>(colsum), out, s));
  return to_status(enqueue_mean_rows(x, n, d, sel, m, out, s));
}

garfield_status garfield_multikrum_noalloc(const float* x, int n, int f, int64_t d, int m,
                                           float* out, int32_t* sel, void* stream) {
  garfield_status st = check_common(x, n, f, d);
  if (st != GARFIELD_OK) return st;
  if (!sel) return GARFIELD_EINVAL;
  if (n < 2 * f + 3) return GARFIELD_EREQ;
  if (m <= 0) m = n - f;
  if (m > n - f) return GARFIELD_EINVAL;
  const DistPlan plan = plan_distances(n, d, x);
  if (dist_workspace_bytes(plan) > GARFIELD_NOALLOC_SCRATCH_BYTES) return GARFIELD_ETOOBIG;
  void* base = nullptr;
  st = static_scratch(&base);
  if (st != GARFIELD_OK) return st;
  hipStream_t s = static_cast<hipStream_t>(stream);
  DistSums ds;
  // every scratch byte a kernel reads here is written earlier in the same call
  // (tile partials, entry sums, probe matrices, reference row), so nothing
  // needs clearing; the mean reads the selected rows (no column sums)
  if (krum_fusable(plan, out)) {
    st = run_distances_on(plan, base, x, 0, &ds, nullptr, s, plan.entries, false);
    if (st != GARFIELD_OK) return st;
    return to_status(enqueue_krum_select_mean(x, ds, d, f, m, sel, out, s));
  }
  st = run_distances_on(plan, base, x, 0, &ds, nullptr, s, kFoldSelect, false);
  if (st != GARFIELD_OK) return st;
  st = to_status(enqueue_krum_select(ds, f, m, sel, s));
  if (st != GARFIELD_OK || !out) return st;
  return to_status(enqueue_mean_rows(x, n, d, sel, m, out, s));
}

garfield_status garfield_krum(const float* x, int n, int f, int64_t d, float* out, int32_t* sel,
                              void* stream) {
  return garfield_multikrum(x, n, f, d, 1, out, sel, stream);
}

garfield_status garfield_multikrum_iterated(const float* x, int n, int f, int64_t d, int m,
                                            float* out, int32_t* sel, void* stream) {
  garfield_status st = check_common(x, n, f, d);
  if (st != GARFIELD_OK) return st;
  if (!sel) return GARFIELD_EINVAL;
  if (n < 2 * f + 3) return GARFIELD_EREQ;
  if (m <= 0) m = n - f;
  if (m > n - f) return GARFIELD_EINVAL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  DistSums ds;
  const bool cs = out && use_colsum(x, n, d, m);
  void* colsum = nullptr;
  st = run_distances(x, n, d, colsum_bytes(cs, d), &ds, &colsum, s, kFoldSelect, cs);
  if (st != GARFIELD_OK) return st;
  st = to_status(enqueue_krum_rounds(ds, f, m, sel, s));
  if (st != GARFIELD_OK || !out) return st;
  if (cs)
    return to_status(enqueue_mean_complement(x, n, d, sel, m, static_cast<double*>(colsum), out, s));
  return to_status(enqueue_mean_rows(x, n, d, sel, m, out, s));
}

garfield_status garfield_median(const float* x, int n, int f, int64_t d, const int32_t* rows,
                                int k, float* out, void* stream) {
  garfield_status st = check_common(x, n, f, d);
  if (st != GARFIELD_OK) return st;
  if (d > 0 && !out) return GARFIELD_EINVAL;
  if (n < 2 * f + 1) return GARFIELD_EREQ;
  if (rows) {
    if (k < 1 || k > n) return GARFIELD_EINVAL;
  } else {
    k = n;
  }
  return to_status(enqueue_median(x, n, d, rows, k, out, static_cast<hipStream_t>(stream)));
}

garfield_status garfield_bulyan(const float* x, int n, int f, int64_t d, float* out,
                                int32_t* sel, void* stream) {
  garfield_status st = check_common(x, n, f, d);
  if (st != GARFIELD_OK) return st;
  if (!sel || (d > 0 && !out)) return GARFIELD_EINVAL;
  if (n < 4 * f + 3) return GARFIELD_EREQ;
  hipStream_t s = static_cast<hipStream_t>(stream);
  DistSums ds;
  st = run_distances(x, n, d, 0, &ds, nullptr, s, kFoldSelect);
  if (st != GARFIELD_OK) return st;
  st = to_status(enqueue_bulyan_select(ds, f, sel, s));
  if (st != GARFIELD_OK) return st;
  return to_status(enqueue_bulyan_aggregate(x, n, f, d, sel, out, s));
}

garfield_status garfield_mda(const float* x, int n, int f, int64_t d, float* out, int32_t* sel,
                             void* stream) {
  garfield_status st = check_common(x, n, f, d);
  if (st != GARFIELD_OK) return st;
  if (!sel) return GARFIELD_EINVAL;
  if (n < 2 * f + 1) return GARFIELD_EREQ;
  const int64_t subsets = binomial(n, f);
  if (subsets < 0 || subsets > GARFIELD_MDA_MAX_SUBSETS) return GARFIELD_ETOOBIG;
  hipStream_t s = static_cast<hipStream_t>(stream);
  void* scratch = nullptr;
  DistSums ds;
  // scratch: the column sums (if used), then the search's per-block results
  const bool cs = out && use_colsum(x, n, d, n - f);
  const size_t cs_bytes = align256(colsum_bytes(cs, d));
  const int fold = mda_uses_cover(n, f) ? kFoldSelect : kFoldMda;
  st = run_distances(x, n, d, cs_bytes + mda_scratch_bytes(n, f), &ds, &scratch, s, fold, cs);
  if (st != GARFIELD_OK) return st;
  st = to_status(enqueue_mda_select(ds, f, static_cast<char*>(scratch) + cs_bytes, sel, s));
  if (st != GARFIELD_OK || !out) return st;
  if (cs)
    return to_status(
        enqueue_mean_complement(x, n, d, sel, n - f, static_cast<double*>(scratch), out, s));
  return to_status(enqueue_mean_rows(x, n, d, sel, n - f, out, s));
}

garfield_status garfield_average(const float* x, int n, int64_t d, float* out, void* stream) {
  garfield_status st = check_common(x, n, 0, d);
  if (st != GARFIELD_OK) return st;
  if (d > 0 && !out) return GARFIELD_EINVAL;
  return to_status(enqueue_mean_rows(x, n, d, nullptr, n, out, static_cast<hipStream_t>(stream)));
}

garfield_status garfield_attack(int kind, const float* honest, int h, int64_t d, double param,
                                uint64_t seed, float* byz, int nbyz, void* stream) {
  if (kind < GARFIELD_ATTACK_REVERSE || kind > GARFIELD_ATTACK_EMPIRE) return GARFIELD_EINVAL;
  if (d < 0 || nbyz < 0 || !std::isfinite(param)) return GARFIELD_EINVAL;
  if (nbyz > GARFIELD_NMAX) return GARFIELD_ETOOBIG;
  const bool uses_honest = kind != GARFIELD_ATTACK_RANDOM;
  if (uses_honest) {
    if (h < 1) return GARFIELD_EINVAL;
    if (h > GARFIELD_NMAX) return GARFIELD_ETOOBIG;
  }
  if (d > 0 && nbyz > 0) {
    if (!byz || reinterpret_cast<uintptr_t>(byz) % sizeof(float) != 0) return GARFIELD_EINVAL;
    if (uses_honest && (!honest || reinterpret_cast<uintptr_t>(honest) % sizeof(float) != 0))
      return GARFIELD_EINVAL;
  }
  return to_status(enqueue_attack(kind, uses_honest ? honest : nullptr, h, d, param, seed, byz,
                                  nbyz, static_cast<hipStream_t>(stream)));
}

garfield_status garfield_variance_stats(const float* g, int h, int64_t d, const float* grad,
                                        double* stats, void* stream) {
  garfield_status st = check_common(g, h, 0, d);
  if (st != GARFIELD_OK) return st;
  if (h < 2 || !stats) return GARFIELD_EINVAL;
  if (d > 0 && (!grad || reinterpret_cast<uintptr_t>(grad) % sizeof(float) != 0))
    return GARFIELD_EINVAL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int64_t parts = d > 0 ? sqnorm_parts(d, grad) : 0;
  DistSums ds;
  void* scratch = nullptr;
  st = run_distances(g, h, d, static_cast<size_t>(parts) * sizeof(double), &ds, &scratch, s);
  if (st != GARFIELD_OK) return st;
  return to_status(
      enqueue_variance_stats(ds, h, grad, d, static_cast<double*>(scratch), stats, s));
}

double garfield_delta(int rule, int n, int f) {
  const double nan = std::nan("");
  if (n < 1 || f < 0) return nan;
  const double nf = static_cast<double>(n - f);
  switch (rule) {
    case GARFIELD_RULE_MDA:
      if (n < 2 * f + 1) return nan;
      return 2.0 * std::sqrt(2.0) * f / nf;
    case GARFIELD_RULE_KRUM:
      if (n < 2 * f + 3) return nan;
      return std::sqrt(2.0 * (nf + (static_cast<double>(f) * (n - f - 2) +
                                    static_cast<double>(f) * f * (n - f - 1)) /
                                       static_cast<double>(n - 2 * f - 2)));
    case GARFIELD_RULE_MEDIAN:
      if (n < 2 * f + 1) return nan;
      return std::sqrt(nf);
    default:
      return nan;
  }
}

double garfield_variance_margin(int rule, int n, int f, const double* stats_host) {
  const double nan = std::nan("");
  const double delta = garfield_delta(rule, n, f);
  if (!stats_host || std::isnan(delta)) return nan;
  const double var = stats_host[0], sq = stats_host[1];
  if (!(var >= 0.0) || !(sq >= 0.0)) return nan;  // also NaN
  const double denom = delta * std::sqrt(var), norm = std::sqrt(sq);
  if (denom == 0.0) return norm > 0.0 ? HUGE_VAL : nan;
  return norm / denom;
}

garfield_status garfield_contract_step(int rule, const float* x, int n, int64_t d,
                                       const int32_t* peers, int q, int f, int m, float* y,
                                       void* stream) {
  garfield_status st = check_common(x, n, f, d);
  if (st != GARFIELD_OK) return st;
  if (!peers || q < 1 || q > n) return GARFIELD_EINVAL;
  if (d > 0 && (!y || reinterpret_cast<uintptr_t>(y) % sizeof(float) != 0)) return GARFIELD_EINVAL;
  switch (rule) {
    case GARFIELD_RULE_KRUM:
    case GARFIELD_RULE_MULTIKRUM:
    case GARFIELD_RULE_MULTIKRUM_ITERATED:
    case GARFIELD_RULE_BULYAN:
    case GARFIELD_RULE_MEDIAN:
    case GARFIELD_RULE_AVERAGE:
    case GARFIELD_RULE_MDA:
      break;
    default:
      return GARFIELD_EINVAL;
  }
  int k = 0;
  st = rule_shape(rule, q, f, &m, &k);  // the rule's requirements apply to the q peers
  if (st != GARFIELD_OK) return st;
  if (rule == GARFIELD_RULE_MDA && binomial(q, f) > GARFIELD_CONTRACT_MDA_MAX_SUBSETS)
    return GARFIELD_ETOOBIG;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (rule == GARFIELD_RULE_MEDIAN)
    return to_status(enqueue_median_nodes(x, n, d, n, peers, q, y, s));
  if (rule == GARFIELD_RULE_AVERAGE)
    return to_status(enqueue_mean_nodes(x, n, d, n, peers, q, y, s));
  DistSums ds;
  void* scratch = nullptr;
  st = run_distances(x, n, d, static_cast<size_t>(n) * k * sizeof(int32_t), &ds, &scratch, s);
  if (st != GARFIELD_OK) return st;
  int32_t* sel = static_cast<int32_t*>(scratch);
  const int rounds = rule == GARFIELD_RULE_BULYAN ? q - 2 * f
                     : rule == GARFIELD_RULE_MULTIKRUM_ITERATED ? m : 0;
  hipError_t e = rule == GARFIELD_RULE_MDA ? enqueue_peer_mda(ds, n, peers, q, f, sel, s)
                 : enqueue_peer_select(ds, n, peers, q, f, m, rounds, k, sel, s);
  if (e != hipSuccess) return to_status(e);
  if (rule == GARFIELD_RULE_BULYAN) return to_status(enqueue_bulyan_nodes(x, n, d, n, q, f, sel, y, s));
  return to_status(enqueue_mean_nodes(x, n, d, n, sel, k, y, s));
}

garfield_status garfield_seg_create(int rule, int n, int f, int m, garfield_segmented** out) {
  if (!out) return GARFIELD_EINVAL;
  *out = nullptr;
  int k = 0;
  garfield_status st = rule_shape(rule, n, f, &m, &k);
  if (st != GARFIELD_OK) return st;
  garfield_segmented* seg = new (std::nothrow) garfield_segmented;
  if (!seg) return GARFIELD_ENOMEM;
  seg->rule = rule;
  seg->n = n;
  seg->f = f;
  seg->m = m;
  seg->k = k;
  if (hipGetDevice(&seg->device) != hipSuccess ||
      hipMalloc(&seg->dacc, sizeof(double) * n * n) != hipSuccess ||
      hipMalloc(&seg->sel, sizeof(int32_t) * n) != hipSuccess ||
      hipMemset(seg->dacc, 0, sizeof(double) * n * n) != hipSuccess ||
      hipDeviceSynchronize() != hipSuccess) {
    (void)hipGetLastError();
    if (seg->dacc) (void)hipFree(seg->dacc);
    if (seg->sel) (void)hipFree(seg->sel);
    delete seg;
    return GARFIELD_ENOMEM;
  }
  *out = seg;
  return GARFIELD_OK;
}

garfield_status garfield_seg_reset(garfield_segmented* seg, void* stream) {
  if (!seg) return GARFIELD_EINVAL;
  seg->selected = false;
  return to_status(enqueue_zero_f64(seg->dacc, seg->n * seg->n, static_cast<hipStream_t>(stream)));
}

garfield_status garfield_seg_accumulate(garfield_segmented* seg, const float* x, int64_t d,
                                        void* stream) {
  if (!seg) return GARFIELD_EINVAL;
  garfield_status st = check_common(x, seg->n, seg->f, d);
  if (st != GARFIELD_OK) return st;
  if (seg->k == 0) return GARFIELD_OK;  // Median and Average use no distances
  hipStream_t s = static_cast<hipStream_t>(stream);
  DistSums ds;
  st = run_distances(x, seg->n, d, 0, &ds, nullptr, s);
  if (st != GARFIELD_OK) return st;
  return to_status(enqueue_accumulate_dist(ds, seg->dacc, s));
}

garfield_status garfield_seg_select(garfield_segmented* seg, int32_t* sel, void* stream) {
  if (!seg) return GARFIELD_EINVAL;
  if (seg->k == 0) return GARFIELD_OK;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const DistSums ds{seg->dacc, kEngineMatrix, seg->n};
  hipError_t e = hipSuccess;
  switch (seg->rule) {
    case GARFIELD_RULE_KRUM:
    case GARFIELD_RULE_MULTIKRUM:
      e = enqueue_krum_select(ds, seg->f, seg->m, seg->sel, s);
      break;
    case GARFIELD_RULE_MULTIKRUM_ITERATED:
      e = enqueue_krum_rounds(ds, seg->f, seg->m, seg->sel, s);
      break;
    case GARFIELD_RULE_BULYAN:
      e = enqueue_bulyan_select(ds, seg->f, seg->sel, s);
      break;
    default: {  // MDA
      void* scratch = nullptr;
      garfield_status st = workspace(mda_scratch_bytes(seg->n, seg->f), &scratch);
      if (st != GARFIELD_OK) return st;
      e = enqueue_mda_select(ds, seg->f, scratch, seg->sel, s);
      break;
    }
  }
  if (e == hipSuccess && sel)
    e = hipMemcpyAsync(sel, seg->sel, sizeof(int32_t) * seg->k, hipMemcpyDeviceToDevice, s);
  if (e == hipSuccess) seg->selected = true;
  return to_status(e);
}

garfield_status garfield_seg_aggregate(garfield_segmented* seg, const float* x, int64_t d,
                                       float* out, void* stream) {
  if (!seg) return GARFIELD_EINVAL;
  garfield_status st = check_common(x, seg->n, seg->f, d);
  if (st != GARFIELD_OK) return st;
  if (d > 0 && !out) return GARFIELD_EINVAL;
  if (seg->k > 0 && !seg->selected) return GARFIELD_EINVAL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int n = seg->n;
  switch (seg->rule) {
    case GARFIELD_RULE_KRUM:
    case GARFIELD_RULE_MULTIKRUM:
    case GARFIELD_RULE_MULTIKRUM_ITERATED:
    case GARFIELD_RULE_MDA:
      return to_status(enqueue_mean_rows(x, n, d, seg->sel, seg->k, out, s));
    case GARFIELD_RULE_BULYAN:
      return to_status(enqueue_bulyan_aggregate(x, n, seg->f, d, seg->sel, out, s));
    case GARFIELD_RULE_MEDIAN:
      return to_status(enqueue_median(x, n, d, nullptr, n, out, s));
    default:  // Average
      return to_status(enqueue_mean_rows(x, n, d, nullptr, n, out, s));
  }
}

// Checks shared by the segment-table calls.
static garfield_status check_table(const garfield_segmented* seg, const float* const* ptrs,
                            const int64_t* dims, int K) {
  if (!seg || K < 0 || (K > 0 && (!ptrs || !dims))) return GARFIELD_EINVAL;
  for (int s = 0; s < K; ++s)
    if (dims[s] < 0) return GARFIELD_EINVAL;
  return GARFIELD_OK;
}

garfield_status garfield_seg_accumulate_table(garfield_segmented* seg, const float* const* ptrs,
                                              const int64_t* dims, int K, void* stream) {
  garfield_status st = check_table(seg, ptrs, dims, K);
  if (st != GARFIELD_OK) return st;
  if (seg->k == 0 || seg->n < 2) return GARFIELD_OK;  // no distances (Median, Average, n = 1)
  // n <= 20: the direct engine; above, the Gram engine over the table
  const bool gram = seg->n > GARFIELD_DIRECT_MAX_N_LIMIT;
  const int64_t tiles = gram ? table_gram_tiles(dims, K, seg->n) : table_tiles(dims, K, seg->n);
  if (tiles < 0) return GARFIELD_ETOOBIG;
  if (tiles == 0) return GARFIELD_OK;  // every segment is empty: all distances 0
  const int nb = (seg->n + 15) / 16;
  const int entries = gram ? nb * (nb + 1) / 2 * 256 : seg->n * (seg->n - 1) / 2;
  void* base = nullptr;
  const size_t partial_bytes = align256(static_cast<size_t>(tiles) * entries * sizeof(double));
  const size_t sums_bytes = align256(entries * sizeof(double));
  st = workspace(partial_bytes + sums_bytes + (gram ? table_gram_probe_bytes() : 0), &base);
  if (st != GARFIELD_OK) return st;
  double* partial = static_cast<double*>(base);
  double* sums = reinterpret_cast<double*>(static_cast<char*>(base) + partial_bytes);
  void* probe = static_cast<char*>(base) + partial_bytes + sums_bytes;
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = gram ? enqueue_distances_table_gram(ptrs, seg->n, dims, K, partial, tiles, probe, s)
                      : enqueue_distances_table(ptrs, seg->n, dims, K, partial, tiles, s);
  if (e == hipSuccess) e = enqueue_sum_tiles(partial, tiles, entries, sums, s);
  if (e == hipSuccess)
    e = enqueue_accumulate_dist(DistSums{sums, gram ? kEngineGram : kEngineDirect, seg->n},
                                seg->dacc, s);
  return to_status(e);
}

garfield_status garfield_seg_aggregate_table(garfield_segmented* seg, const float* const* ptrs,
                                             const int64_t* dims, int K, float* const* outs,
                                             void* stream) {
  garfield_status st = check_table(seg, ptrs, dims, K);
  if (st != GARFIELD_OK) return st;
  if (K > 0 && !outs) return GARFIELD_EINVAL;
  for (int s = 0; s < K; ++s)
    if (dims[s] > 0 && (!outs[s] || reinterpret_cast<uintptr_t>(outs[s]) % sizeof(float) != 0))
      return GARFIELD_EINVAL;
  if (seg->k > 0 && !seg->selected) return GARFIELD_EINVAL;
  hipStream_t s = static_cast<hipStream_t>(stream);
  const int n = seg->n;
  switch (seg->rule) {
    case GARFIELD_RULE_KRUM:
    case GARFIELD_RULE_MULTIKRUM:
    case GARFIELD_RULE_MULTIKRUM_ITERATED:
    case GARFIELD_RULE_MDA:
      return to_status(enqueue_mean_rows_table(ptrs, n, dims, outs, K, seg->sel, seg->k, s));
    case GARFIELD_RULE_BULYAN:
      return to_status(enqueue_bulyan_table(ptrs, n, seg->f, dims, outs, K, seg->sel, s));
    case GARFIELD_RULE_MEDIAN:
      return to_status(enqueue_median_table(ptrs, n, dims, outs, K, s));
    default:  // Average
      return to_status(enqueue_mean_rows_table(ptrs, n, dims, outs, K, nullptr, n, s));
  }
}

garfield_status garfield_seg_destroy(garfield_segmented* seg) {
  if (!seg) return GARFIELD_OK;
  int cur = 0;
  (void)hipGetDevice(&cur);
  (void)hipSetDevice(seg->device);
  const hipError_t e = hipDeviceSynchronize();
  (void)hipFree(seg->dacc);
  (void)hipFree(seg->sel);
  (void)hipSetDevice(cur);
  delete seg;
  return to_status(e);
}

size_t garfield_workspace_bytes(int rule, int n, int f, int64_t d, int m) {
  if (n < 1 || n > GARFIELD_NMAX || f < 0 || d < 0) return 0;
  // Plan for float-aligned rows, as every accepted input is: the same plan as
  // every call of the rule with these sizes.
  const float* narrow = reinterpret_cast<const float*>(uintptr_t{4});
  switch (rule) {
    case GARFIELD_RULE_MULTIKRUM:
    case GARFIELD_RULE_MULTIKRUM_ITERATED: {
      const int mm = m <= 0 ? n - f : m;
      return dist_workspace_bytes(plan_distances(n, d, narrow)) +
             align256(colsum_bytes(use_colsum(narrow, n, d, mm), d));
    }
    case GARFIELD_RULE_DIST:
    case GARFIELD_RULE_KRUM:
    case GARFIELD_RULE_BULYAN:
      return dist_workspace_bytes(plan_distances(n, d, narrow));
    case GARFIELD_RULE_MDA: {
      const int64_t subsets = binomial(n, f);
      if (n < 2 * f + 1 || subsets < 0 || subsets > GARFIELD_MDA_MAX_SUBSETS) return 0;
      return dist_workspace_bytes(plan_distances(n, d, narrow)) +
             align256(colsum_bytes(use_colsum(narrow, n, d, n - f), d)) +
             align256(mda_scratch_bytes(n, f));
    }
    case GARFIELD_RULE_MEDIAN:
    case GARFIELD_RULE_AVERAGE:
      return 0;
    default:
      return 0;
  }
}

garfield_status garfield_release(void) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return to_status(hipErrorInvalidDevice);
  std::lock_guard<std::mutex> lock(g_mutex);
  auto it = g_workspaces.find(dev);
  if (it == g_workspaces.end() || !it->second.ptr) return GARFIELD_OK;
  if (hipDeviceSynchronize() != hipSuccess) return to_status(hipErrorUnknown);
  (void)hipFree(it->second.ptr);
  g_workspaces.erase(it);
  return GARFIELD_OK;
}

const char* garfield_strerror(garfield_status s) {
  switch (s) {
    case GARFIELD_OK: return "success";
    case GARFIELD_EINVAL: return "invalid argument (null pointer, n < 1, f < 0, d < 0, m or k out of range)";
    case GARFIELD_EREQ: return "n is below the rule's requirement in f";
    case GARFIELD_ETOOBIG: return "problem too large (n > GARFIELD_NMAX, too many MDA subsets, or d beyond one launch)";
    case GARFIELD_ENOMEM: return "device workspace allocation failed";
    case GARFIELD_EHIP: return "HIP runtime error";
  }
  return "unknown status";
}

const char* garfield_version(void) { return "garfield-mi355x 0.1"; }

int garfield_tuning_set_direct_max_n(int n) {
  if (n < 1 || n > GARFIELD_DIRECT_MAX_N_LIMIT) return -1;
  const int old = direct_max_n();
  set_direct_max_n(n);
  return old;
}

long long garfield_tuning_set_mda_cover_min(long long subsets) {
  const long long old = mda_cover_min();
  if (subsets >= 0) set_mda_cover_min(subsets);
  return old;
}

int garfield_tuning_set_stream_residency(int wgs_per_cu) {
  const int old = stream_residency();
  set_stream_residency(wgs_per_cu < 0 ? -1 : wgs_per_cu);
  return old;
}

int garfield_tuning_set_fused(int on) {
  const int old = fused_enabled() ? 1 : 0;
  set_fused(on != 0);
  return old;
}

int garfield_tuning_gram_reference(const float* x, int n, long long d, void* stream) {
  if (check_common(x, n, 0, d) != GARFIELD_OK || n < 2 || d < 1) return -1;
  DistPlan plan = plan_distances(n, d, x);
  plan.engine = kEngineGram;
  hipStream_t s = static_cast<hipStream_t>(stream);
  void* base = nullptr;
  if (workspace(dist_workspace_bytes(plan), &base) != GARFIELD_OK) return -1;
  const DistWorkspace ws = carve_dist_workspace(plan, base);
  if (enqueue_reference(x, plan, ws, s) != hipSuccess) return -1;
  int32_t ref = -1;
  if (hipMemcpyAsync(&ref, ws.ref, sizeof(ref), hipMemcpyDeviceToHost, s) != hipSuccess) return -1;
  if (hipStreamSynchronize(s) != hipSuccess) return -1;
  return ref;
}

int garfield_tuning_table_gram_reference(const float* const* ptrs, int n, const long long* dims,
                                         int K, void* stream) {
  if (!ptrs || !dims || n < 2 || n > GARFIELD_NMAX || K < 1) return -1;
  for (int k = 0; k < K; ++k)
    if (dims[k] < 0) return -1;
  std::vector<int64_t> d64(dims, dims + K);
  hipStream_t s = static_cast<hipStream_t>(stream);
  void* base = nullptr;
  if (workspace(table_gram_probe_bytes(), &base) != GARFIELD_OK) return -1;
  if (enqueue_table_reference(ptrs, n, d64.data(), K, base, s) != hipSuccess) return -1;
  int32_t ref = -1;
  if (hipMemcpyAsync(&ref, table_reference_slot(base), sizeof(ref), hipMemcpyDeviceToHost, s) !=
      hipSuccess)
    return -1;
  if (hipStreamSynchronize(s) != hipSuccess) return -1;
  return ref;
}

int garfield_tuning_set_kernel_timing(int on) {
  const int old = timing_enabled() ? 1 : 0;
  timing_set(on != 0);
  return old;
}

size_t garfield_tuning_kernel_timing(char* buf, size_t len) { return timing_summary(buf, len); }

int garfield_tuning_stream_read(const float* x, long long count, float* sums, void* stream) {
  if (!x || !sums || count < 0 || count % 4 != 0 || reinterpret_cast<uintptr_t>(x) % 16 != 0 ||
      reinterpret_cast<uintptr_t>(sums) % sizeof(float) != 0)
    return GARFIELD_EINVAL;
  return to_status(enqueue_stream_read(x, count, GARFIELD_TUNING_READ_BLOCKS, sums,
                                       static_cast<hipStream_t>(stream)));
}

int garfield_tuning_distance_engine(int n, long long d) {
  if (n < 1 || n > GARFIELD_NMAX || d < 0) return -1;
  const float* aligned = reinterpret_cast<const float*>(uintptr_t{256});
  return plan_distances(n, d, aligned).engine;
}

}  // extern "C"
