// Streaming per-coordinate aggregation over HBM: one pass over the k rows an
// aggregate needs, one write of d floats.
//
//  * mean of a row subset (Multi-Krum, MDA, Average; Krum is the 1-row case):
//    fp64 sums in ascending row order, one rounding to fp32 at the end;
//  * coordinate-wise median (Section 3.1 item 1): a branch-free selection
//    network on k registers per coordinate (the paper's GPU median is built on
//    a branchless 3-element sort, Section 4.3; on CDNA the min/max/med3
//    instructions play that role and a pruned odd-even merge network replaces
//    the selection loop);
//  * Bulyan's aggregation (Section 3.1 item 4): a full sorting network on the
//    theta selected values, the median, then the beta values closest to it
//    under the key (|v - median|, v) -- in sorted order these form a window
//    around the middle whose split is found by beta comparisons -- averaged.
//
// Row indices come from device memory (the selection kernels write them), so
// no host round trip separates selection from aggregation.

#include <map>
#include <mutex>
#include <set>
#include <utility>

#include "aggregate_body.h"
#include "device_common.h"
#include "internal.h"
#include "timing.h"

namespace garfield {

namespace {

// The kernels over one row-major n x d matrix; the per-coordinate work is in
// aggregate_body.h (shared with the segment-table kernels).
// LISTED: the rows listed in `rows` (ListedRows), else rows 0 .. k-1.
template <int W, bool LISTED>
__global__ __launch_bounds__(kBlock) void k_mean_rows(const float* __restrict__ x, int n,
                                                      int64_t d, const int32_t* __restrict__ rows,
                                                      int k, float* __restrict__ out) {
  const MatrixRows src{x, d};
  const int64_t c = (static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x) * W;
  if (c >= d) return;
  if constexpr (LISTED) mean_at<W>(src, d, ListedRows{rows, n}, k, c, out);
  else mean_at<W>(src, d, AllRows{}, k, c, out);
}

// Mean of the k distinct rows of sel from the distance step's column sums
// (enqueue_mean_complement): thread 0 lists the rows not in sel, ascending, in
// LDS; every lane subtracts them from its coordinates' column sums where all
// W of those are exact (not NaN), and otherwise sums the rows of sel as
// k_mean_rows does. Either way the fp64 value is the exact sum k_mean_rows
// forms (sums of these values are exact where the column sum is), rounded
// once.
template <int W>
__global__ __launch_bounds__(kBlock) void k_mean_complement(const float* __restrict__ x, int n,
                                                            int64_t d,
                                                            const int32_t* __restrict__ sel, int k,
                                                            const double* __restrict__ colsum,
                                                            float* __restrict__ out) {
  __shared__ int32_t rest[kNmax];
  __shared__ int nrest;
  if (threadIdx.x == 0) {
    uint64_t mask = 0;
    for (int t = 0; t < k; ++t) mask |= uint64_t{1} << row_of(sel, t, n);
    int q = 0;
    for (int r = 0; r < n; ++r)
      if (!((mask >> r) & 1)) rest[q++] = r;
    nrest = q;
  }
  __syncthreads();
  const int q = nrest;
  const MatrixRows src{x, d};
  const double count = static_cast<double>(k);
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock * W;
  for (int64_t c = (static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x) * W; c < d;
       c += stride) {
    const bool full = c + W <= d;
    double acc[W];
    bool loaded = false;
    if constexpr (W >= 2) {
      if (full) {  // ordinary 16-byte loads: a line's halves meet in L2
#pragma unroll
        for (int e = 0; e < W; e += 2) {
          const d2 t = *reinterpret_cast<const d2*>(colsum + c + e);
          acc[e] = t.x;
          acc[e + 1] = t.y;
        }
        loaded = true;
      }
    }
    if (!loaded) {
#pragma unroll
      for (int e = 0; e < W; ++e) acc[e] = (c + e < d) ? colsum[c + e] : 0.0;
    }
    bool exact = true;
#pragma unroll
    for (int e = 0; e < W; ++e) exact = exact && !__builtin_isnan(acc[e]);
    if (exact) {
      for (int t = 0; t < q; t += 2) {  // two rows' loads in flight
        const bool two = t + 1 < q;
        float v[2][W];
        const float* p0 = src.row(rest[t]) + c;
        const float* p1 = src.row(rest[two ? t + 1 : t]) + c;
        if (full) {
          load_w<W>(p0, v[0]);
          load_w<W>(p1, v[1]);
        } else {
          load_w_tail<W>(p0, d - c, v[0]);
          load_w_tail<W>(p1, d - c, v[1]);
        }
#pragma unroll
        for (int e = 0; e < W; ++e) acc[e] -= static_cast<double>(v[0][e]);
        if (two) {
#pragma unroll
          for (int e = 0; e < W; ++e) acc[e] -= static_cast<double>(v[1][e]);
        }
      }
    } else {
#pragma unroll
      for (int e = 0; e < W; ++e) acc[e] = 0.0;
      if (full) sum_rows_at<W, true, true>(src, d, ListedRows{sel, n}, k, c, acc);
      else sum_rows_at<W, false, true>(src, d, ListedRows{sel, n}, k, c, acc);
    }
    float o[W];
#pragma unroll
    for (int e = 0; e < W; ++e) o[e] = static_cast<float>(acc[e] / count);
    store_out<W>(out, c, d, full, o);
  }
}

// ---------------------------------------------------------------------------
// Every lane loads W consecutive coordinates of each of the K rows: 16-byte
// loads (W = 4) stream a K-row gather far faster than 8- or 4-byte ones, so
// W = 4 is kept up to K = kMedianX4MaxK, where the K x 4 values still fit the
// registers of two waves per SIMD.
constexpr int kMedianX4MaxK = 52;

template <int K, int W, bool LISTED>
__global__ __launch_bounds__(kBlock) void k_median(const float* __restrict__ x, int n, int64_t d,
                                                   const int32_t* __restrict__ rows,
                                                   float* __restrict__ out) {
  const MatrixRows src{x, d};
  const int64_t c = (static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x) * W;
  if (c >= d) return;
  if constexpr (LISTED) median_at<K, W>(src, d, ListedRows{rows, n}, c, out);
  else median_at<K, W>(src, d, AllRows{}, c, out);
}

// Bulyan aggregation for theta = T selected rows (bulyan_at); the sorted
// column of each thread goes through LDS.
template <int T, int W>
__global__ __launch_bounds__(kBlock) void k_bulyan_agg(const float* __restrict__ x, int n,
                                                       int64_t d, const int32_t* __restrict__ sel,
                                                       int beta, float* __restrict__ out) {
  __shared__ float sorted[T * kBlock];
  const MatrixRows src{x, d};
  const int64_t c = (static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x) * W;
  if (c < d) bulyan_at<T, W>(src, d, ListedRows{sel, n}, beta, c, sorted + threadIdx.x, out);
}

// Residency of the gathers. Each lane issues its rows' loads back to back;
// with as many workgroups per CU as the registers allow, so many loads are in
// flight that HBM serves them less well. Measured on the median (W = 4, k = 5
// to 35 rows of 25.6 M floats) and on Bulyan's band path (T = 5 to 19), two to
// four workgroups per CU -- about 100 to 140 KB of loads in flight per CU --
// stream 3 to 10 % faster than no cap (k = 11: 0.728 -> 0.773 of 8 TB/s,
// T = 11: 0.711 -> 0.763); the mean (whose lanes also divide in fp64),
// Bulyan's general LDS path and the 2-float paths lose with a cap, and the
// 49-row median is held at two by its registers anyway. The cap is set by
// reserving LDS that the kernels never touch.
int g_stream_cap = 0;  // 0: each kernel's rule; > 0: that many workgroups per CU; < 0: none

// The rule: the number of workgroups whose in-flight loads come nearest
// `target` bytes per CU from below, between 2 and 4.
int cap_for(int64_t inflight, int64_t target) {
  const int64_t c = target / inflight;
  return c < 2 ? 2 : (c > 4 ? 4 : static_cast<int>(c));
}

std::mutex g_lds_mutex;
std::map<int, int> g_lds_per_cu;        // device -> LDS bytes per CU
std::set<std::pair<int, const void*>> g_lds_raised;  // (device, kernel) allowed > 64 KB

int lds_per_cu(int dev) {
  std::lock_guard<std::mutex> lock(g_lds_mutex);
  auto it = g_lds_per_cu.find(dev);
  if (it != g_lds_per_cu.end()) return it->second;
  int v = 0;
  if (hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, dev) !=
          hipSuccess || v <= 0) {
    (void)hipGetLastError();
    v = 160 * 1024;
  }
  g_lds_per_cu.emplace(dev, v);
  return v;
}

// Dynamic LDS for a launch of `kernel` (static LDS static_lds bytes) that
// holds it to rule_cap workgroups per CU (none if negative), unless the
// tuning setting overrides the rule; 0 when no cap applies. *e receives an
// error of the attribute call, if any.
size_t residency_lds(const void* kernel, size_t static_lds, int rule_cap, hipError_t* e) {
  *e = hipSuccess;
  const int set = __atomic_load_n(&g_stream_cap, __ATOMIC_RELAXED);
  const int cap = set == 0 ? rule_cap : set;
  if (cap <= 0) return 0;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) {
    (void)hipGetLastError();
    return 0;
  }
  const size_t per_cu = static_cast<size_t>(lds_per_cu(dev));
  // just over a (cap + 1)-th of the CU's LDS: at most `cap` workgroups fit
  const size_t want = per_cu / (cap + 1) + 1024;
  const size_t dyn = want > static_lds ? want - static_lds : 0;
  if (dyn > 65536) {
    std::lock_guard<std::mutex> lock(g_lds_mutex);
    if (!g_lds_raised.count({dev, kernel})) {
      *e = hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                               static_cast<int>(dyn));
      if (*e != hipSuccess) return 0;
      g_lds_raised.insert({dev, kernel});
    }
  }
  return dyn;
}

template <typename K>
size_t static_lds_of(K kernel) {
  hipFuncAttributes a{};
  if (hipFuncGetAttributes(&a, reinterpret_cast<const void*>(kernel)) != hipSuccess) {
    (void)hipGetLastError();
    return 0;
  }
  return a.sharedSizeBytes;
}

// ---------------------------------------------------------------------------
// One pass: a workgroup per kBlock items, so every lane handles one item. A
// single pass streams measurably faster than a capped grid looping over d,
// and the gathers have no loop to hoist their per-row address arithmetic out
// of (where it would hold one register pair per row). 2^31 - 1 workgroups of
// kBlock lanes cover any d a device holds; beyond them grid_for returns 0 and
// the launch is refused (mean_complement alone still loops).
int grid_for(int64_t items) {
  const int64_t blocks = (items + kBlock - 1) / kBlock;
  if (blocks > 0x7fffffff) return 0;
  return blocks < 1 ? 1 : static_cast<int>(blocks);
}

template <int W>
hipError_t launch_mean(const float* x, int n, int64_t d, const int32_t* rows, int k, float* out,
                       hipStream_t s) {
  const int grid = grid_for((d + W - 1) / W);
  if (grid == 0) return hipErrorInvalidValue;
  if (rows)
    launch("mean_rows", k_mean_rows<W, true>, dim3(grid), dim3(kBlock), 0, s, x, n, d, rows, k,
           out);
  else
    launch("mean_rows", k_mean_rows<W, false>, dim3(grid), dim3(kBlock), 0, s, x, n, d, rows, k,
           out);
  return hipGetLastError();
}

template <int W>
hipError_t launch_mean_complement(const float* x, int n, int64_t d, const int32_t* sel, int k,
                                  const double* colsum, float* out, hipStream_t s) {
  const int grid = grid_for((d + W - 1) / W);
  if (grid == 0) return hipErrorInvalidValue;
  launch("mean_complement", k_mean_complement<W>, dim3(grid), dim3(kBlock), 0,
         s, x, n, d, sel, k, colsum, out);
  return hipGetLastError();
}

template <int K, int W, bool LISTED>
hipError_t launch_median_kwl(const float* x, int n, int64_t d, const int32_t* rows, float* out,
                             hipStream_t s) {
  hipError_t e;
  const int rule = W == 4 ? cap_for(int64_t{kBlock} * W * 4 * K, 100 * 1024) : -1;
  const size_t lds =
      residency_lds(reinterpret_cast<const void*>(k_median<K, W, LISTED>), 0, rule, &e);
  if (e != hipSuccess) return e;
  const int grid = grid_for((d + W - 1) / W);
  if (grid == 0) return hipErrorInvalidValue;
  launch("median", k_median<K, W, LISTED>, dim3(grid), dim3(kBlock), static_cast<uint32_t>(lds),
         s, x, n, d, rows, out);
  return hipGetLastError();
}

template <int K, int W>
hipError_t launch_median_kw(const float* x, int n, int64_t d, const int32_t* rows, float* out,
                            hipStream_t s) {
  if (rows) return launch_median_kwl<K, W, true>(x, n, d, rows, out, s);
  return launch_median_kwl<K, W, false>(x, n, d, rows, out, s);
}

template <int K>
hipError_t launch_median_k(int width, const float* x, int n, int64_t d, const int32_t* rows,
                           float* out, hipStream_t s) {
  if constexpr (K <= kMedianX4MaxK) {
    if (width == 4) return launch_median_kw<K, 4>(x, n, d, rows, out, s);
  }
  if (width >= 2) return launch_median_kw<K, 2>(x, n, d, rows, out, s);
  return launch_median_kw<K, 1>(x, n, d, rows, out, s);
}

template <int K>
hipError_t median_dispatch(int k, int width, const float* x, int n, int64_t d,
                           const int32_t* rows, float* out, hipStream_t s) {
  if constexpr (K > kNmax) {
    return hipErrorInvalidValue;
  } else {
    if (k == K) return launch_median_k<K>(width, x, n, d, rows, out, s);
    return median_dispatch<K + 1>(k, width, x, n, d, rows, out, s);
  }
}

template <int T, int W>
hipError_t launch_bulyan_tw(int beta, const float* x, int n, int64_t d, const int32_t* sel,
                            float* out, hipStream_t s) {
  static const size_t static_lds = static_lds_of(k_bulyan_agg<T, W>);
  hipError_t e;
  // the band path only (beta = 3, odd theta: registers, no LDS column)
  const int rule = (W == 4 && beta == 3 && T % 2 == 1) ? cap_for(int64_t{kBlock} * W * 4 * T, 140 * 1024)
                                                        : -1;
  const size_t lds =
      residency_lds(reinterpret_cast<const void*>(k_bulyan_agg<T, W>), static_lds, rule, &e);
  if (e != hipSuccess) return e;
  const int grid = grid_for((d + W - 1) / W);
  if (grid == 0) return hipErrorInvalidValue;
  launch("bulyan_agg", k_bulyan_agg<T, W>, dim3(grid), dim3(kBlock), static_cast<uint32_t>(lds), s,
         x, n, d, sel, beta, out);
  return hipGetLastError();
}

template <int T>
hipError_t bulyan_dispatch(int theta, int beta, int width, const float* x, int n, int64_t d,
                           const int32_t* sel, float* out, hipStream_t s) {
  if constexpr (T > kNmax) {
    return hipErrorInvalidValue;
  } else {
    if (theta == T) {
      if constexpr (T <= 24) {
        if (width == 4) return launch_bulyan_tw<T, 4>(beta, x, n, d, sel, out, s);
      }
      if constexpr (T <= 48) {
        if (width >= 2) return launch_bulyan_tw<T, 2>(beta, x, n, d, sel, out, s);
      }
      return launch_bulyan_tw<T, 1>(beta, x, n, d, sel, out, s);
    }
    return bulyan_dispatch<T + 1>(theta, beta, width, x, n, d, sel, out, s);
  }
}

}  // namespace

// Load/store width of the streaming kernels: 16-byte accesses whenever x and
// out are float-aligned, whatever d (see f4u); one float at a time only for
// an output that is not float-aligned.
int stream_width(const float* x, const float* out) {
  return (load_width(x) == 4 && load_width(out) == 4) ? 4 : 1;
}

int stream_residency() { return __atomic_load_n(&g_stream_cap, __ATOMIC_RELAXED); }
void set_stream_residency(int wgs_per_cu) {
  __atomic_store_n(&g_stream_cap, wgs_per_cu, __ATOMIC_RELAXED);
}

hipError_t enqueue_mean_rows(const float* x, int n, int64_t d, const int32_t* rows, int k,
                             float* out, hipStream_t s) {
  if (d == 0) return hipSuccess;
  const int w = stream_width(x, out);
  if (w == 4) return launch_mean<4>(x, n, d, rows, k, out, s);
  if (w == 2) return launch_mean<2>(x, n, d, rows, k, out, s);
  return launch_mean<1>(x, n, d, rows, k, out, s);
}

hipError_t enqueue_mean_complement(const float* x, int n, int64_t d, const int32_t* sel, int k,
                                   const double* colsum, float* out, hipStream_t s) {
  if (d == 0) return hipSuccess;
  if (n < 1 || n > kNmax || k < 1 || !sel || !colsum) return hipErrorInvalidValue;
  const int w = stream_width(x, out);
  if (w == 4) return launch_mean_complement<4>(x, n, d, sel, k, colsum, out, s);
  return launch_mean_complement<1>(x, n, d, sel, k, colsum, out, s);
}

hipError_t enqueue_median(const float* x, int n, int64_t d, const int32_t* rows, int k,
                          float* out, hipStream_t s) {
  if (d == 0) return hipSuccess;
  return median_dispatch<1>(k, stream_width(x, out), x, n, d, rows, out, s);
}

hipError_t enqueue_bulyan_aggregate(const float* x, int n, int f, int64_t d, const int32_t* sel,
                                    float* out, hipStream_t s) {
  if (d == 0) return hipSuccess;
  const int theta = n - 2 * f;
  const int beta = theta - 2 * f;
  return bulyan_dispatch<1>(theta, beta, stream_width(x, out), x, n, d, sel, out, s);
}

namespace {

// Read-rate probe: workgroup b sums the float4s b*kBlock*4 + t + u*kBlock
// (u < 4), then the same a grid's worth further on, with nontemporal loads,
// and writes the workgroup's fp32 total.
__global__ __launch_bounds__(kBlock) void k_stream_read(const f4* __restrict__ x, int64_t m,
                                                        float* __restrict__ sums) {
  constexpr int U = 4;
  __shared__ float red[kBlock];
  float acc = 0.0f;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock * U;
  for (int64_t base = static_cast<int64_t>(blockIdx.x) * kBlock * U + threadIdx.x; base < m;
       base += stride) {
    f4 v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t i = base + static_cast<int64_t>(u) * kBlock;
      v[u] = i < m ? __builtin_nontemporal_load(x + i) : f4{0.0f, 0.0f, 0.0f, 0.0f};
    }
#pragma unroll
    for (int u = 0; u < U; ++u) acc += (v[u].x + v[u].y) + (v[u].z + v[u].w);
  }
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int h = kBlock / 2; h > 0; h >>= 1) {
    if (static_cast<int>(threadIdx.x) < h) red[threadIdx.x] += red[threadIdx.x + h];
    __syncthreads();
  }
  if (threadIdx.x == 0) sums[blockIdx.x] = red[0];
}

}  // namespace

hipError_t enqueue_stream_read(const float* x, int64_t count, int blocks, float* sums,
                               hipStream_t s) {
  launch("stream_read", k_stream_read, dim3(blocks), dim3(kBlock), 0, s,
         reinterpret_cast<const f4*>(x), count / 4, sums);
  return hipGetLastError();
}

}  // namespace garfield
