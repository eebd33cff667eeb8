// Segment tables: the n vectors given as K segments stored apart -- each
// layer's gradient from each of n workers (per-layer aggregation, Section
// 4.2), or n whole vectors in separate buffers (K = 1). ptrs[s * n + i] points
// to segment s of vector i (dims[s] floats). One launch streams every segment
// of a batch: workgroup b finds its segment by a search over the segments'
// first workgroups (rows.h), so K small segments cost one launch, not K. The
// per-coordinate work is the matrix kernels' own (direct_body.h,
// aggregate_body.h); only the addressing differs.

#include "aggregate_body.h"
#include "direct_body.h"
#include "internal.h"
#include "timing.h"

namespace garfield {

namespace {

// Distances: a segment's tiles are consecutive, span[s] coordinates each (the
// matrix engine's tile for that length, direct_chunk); tile b of this launch
// writes column tile_base + b of the entry-major partials.
template <int N, int W>
__global__ __launch_bounds__(kBlock) void k_dist_direct_seg(const float* const* __restrict__ ptrs,
                                                             SegTable tab, int64_t tile_base,
                                                             int64_t tiles,
                                                             double* __restrict__ partial) {
  constexpr int P = N * (N - 1) / 2;
  float acc[P];
#pragma unroll
  for (int p = 0; p < P; ++p) acc[p] = 0.0f;
  const int b = blockIdx.x;
  const int s = seg_of(tab, b);
  const int64_t start = static_cast<int64_t>(b - tab.first[s]) * tab.span[s];
  const int64_t d = tab.dims[s];
  const int64_t end = start + tab.span[s] < d ? start + tab.span[s] : d;
  direct_accumulate<N, W>(TableRows{ptrs + static_cast<int64_t>(s) * N}, start, end, acc);
  block_reduce_pairs<P>(acc, partial + tile_base + b, tiles);
}

// Aggregation: workgroup b covers kBlock * W coordinates of its segment (the
// mean: W = 4; median and Bulyan: W by the row count, as in the matrix kernels).
constexpr auto kAggSpan = [](int64_t) { return static_cast<int64_t>(kBlock) * 4; };
template <int W>
__device__ __forceinline__ int64_t seg_coord(const SegTable& tab, int s, int b) {
  return (static_cast<int64_t>(b - tab.first[s]) * kBlock + threadIdx.x) * W;
}

// LISTED: the rows listed in `rows`, else rows 0 .. k-1.
template <int W, bool LISTED>
__global__ __launch_bounds__(kBlock) void k_mean_rows_seg(const float* const* __restrict__ ptrs,
                                                          int n, const int32_t* __restrict__ rows,
                                                          int k, SegTable tab) {
  const int s = seg_of(tab, blockIdx.x);
  const int64_t c = seg_coord<W>(tab, s, blockIdx.x);
  if (c >= tab.dims[s]) return;
  const TableRows src{ptrs + static_cast<int64_t>(s) * n};
  if constexpr (LISTED) mean_at<W>(src, tab.dims[s], ListedRows{rows, n}, k, c, tab.outs[s]);
  else mean_at<W>(src, tab.dims[s], AllRows{}, k, c, tab.outs[s]);
}

// The median over all K = n vectors of each segment.
template <int K, int W>
__global__ __launch_bounds__(kBlock) void k_median_seg(const float* const* __restrict__ ptrs,
                                                       SegTable tab) {
  const int s = seg_of(tab, blockIdx.x);
  const int64_t c = seg_coord<W>(tab, s, blockIdx.x);
  if (c < tab.dims[s])
    median_at<K, W>(TableRows{ptrs + static_cast<int64_t>(s) * K}, tab.dims[s], AllRows{}, c,
                    tab.outs[s]);
}

template <int T, int W>
__global__ __launch_bounds__(kBlock) void k_bulyan_agg_seg(const float* const* __restrict__ ptrs,
                                                           int n, const int32_t* __restrict__ sel,
                                                           int beta, SegTable tab) {
  __shared__ float sorted[T * kBlock];
  const int s = seg_of(tab, blockIdx.x);
  const int64_t c = seg_coord<W>(tab, s, blockIdx.x);
  if (c < tab.dims[s])
    bulyan_at<T, W>(TableRows{ptrs + static_cast<int64_t>(s) * n}, tab.dims[s],
                    ListedRows{sel, n}, beta, c, sorted + threadIdx.x, tab.outs[s]);
}

// Cut a batch of K segments into launches of at most kSegMax segments and
// call f(first segment, table, workgroups) for each launch that has work;
// per(d) = coordinates per workgroup for a segment of length d.
template <class Per, class F>
hipError_t for_each_launch(const int64_t* dims, float* const* outs, int K, Per&& per, F&& f) {
  for (int g0 = 0; g0 < K; g0 += kSegMax) {
    SegTable tab{};
    tab.count = K - g0 < kSegMax ? K - g0 : kSegMax;
    int64_t total = 0;
    for (int s = 0; s < tab.count; ++s) {
      const int64_t span = per(dims[g0 + s]);
      tab.first[s] = static_cast<int32_t>(total);
      tab.span[s] = static_cast<int32_t>(span);
      tab.dims[s] = dims[g0 + s];
      tab.outs[s] = outs ? outs[g0 + s] : nullptr;
      total += (dims[g0 + s] + span - 1) / span;
      if (total > 0x7fffffff) return hipErrorInvalidValue;
    }
    tab.first[tab.count] = static_cast<int32_t>(total);
    if (total == 0) continue;
    const hipError_t e = f(g0, tab, total);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

template <int N, int W>
hipError_t dist_seg_nw(const float* const* ptrs, const int64_t* dims, int K, double* partial,
                       int64_t tiles, hipStream_t s) {
  int64_t base = 0;
  auto per = [](int64_t d) { return direct_chunk(d, W); };
  return for_each_launch(dims, nullptr, K, per, [&](int g0, const SegTable& tab,
                                                    int64_t total) {
    launch("dist_direct_seg", k_dist_direct_seg<N, W>, dim3(static_cast<unsigned>(total)),
           dim3(kBlock), 0, s, ptrs + static_cast<int64_t>(g0) * N, tab, base, tiles, partial);
    base += total;
    return hipGetLastError();
  });
}

template <int N>
hipError_t dist_seg_dispatch(int n, const float* const* ptrs, const int64_t* dims, int K,
                             double* partial, int64_t tiles, hipStream_t s) {
  if constexpr (N > kDirectMaxNLimit) {
    return hipErrorInvalidValue;
  } else {
    if (n != N) return dist_seg_dispatch<N + 1>(n, ptrs, dims, K, partial, tiles, s);
    // the direct engine's register budget: 16-byte loads up to 12 rows, 8-byte to 19
    if constexpr (N <= 12) return dist_seg_nw<N, 4>(ptrs, dims, K, partial, tiles, s);
    else if constexpr (N <= 19) return dist_seg_nw<N, 2>(ptrs, dims, K, partial, tiles, s);
    else return dist_seg_nw<N, 1>(ptrs, dims, K, partial, tiles, s);
  }
}

// Widths as the matrix kernels choose them: the K (or T) x W values of a lane
// within the registers of two waves per SIMD.
template <int K>
hipError_t median_seg_dispatch(int n, const float* const* ptrs, const int64_t* dims,
                               float* const* outs, int nseg, hipStream_t s) {
  if constexpr (K > kNmax) {
    return hipErrorInvalidValue;
  } else {
    if (n != K) return median_seg_dispatch<K + 1>(n, ptrs, dims, outs, nseg, s);
    constexpr int W = K <= 52 ? 4 : 2;
    auto per = [](int64_t) { return static_cast<int64_t>(kBlock) * W; };
    return for_each_launch(dims, outs, nseg, per, [&](int g0, const SegTable& tab,
                                                      int64_t total) {
      launch("median_seg", k_median_seg<K, W>, dim3(static_cast<unsigned>(total)), dim3(kBlock), 0,
             s, ptrs + static_cast<int64_t>(g0) * K, tab);
      return hipGetLastError();
    });
  }
}

template <int T>
hipError_t bulyan_seg_dispatch(int theta, int beta, const float* const* ptrs, int n,
                               const int32_t* sel, const int64_t* dims, float* const* outs,
                               int nseg, hipStream_t s) {
  if constexpr (T > kNmax) {
    return hipErrorInvalidValue;
  } else {
    if (theta != T)
      return bulyan_seg_dispatch<T + 1>(theta, beta, ptrs, n, sel, dims, outs, nseg, s);
    constexpr int W = T <= 24 ? 4 : (T <= 48 ? 2 : 1);
    auto per = [](int64_t) { return static_cast<int64_t>(kBlock) * W; };
    return for_each_launch(dims, outs, nseg, per, [&](int g0, const SegTable& tab,
                                                      int64_t total) {
      launch("bulyan_agg_seg", k_bulyan_agg_seg<T, W>, dim3(static_cast<unsigned>(total)),
             dim3(kBlock), 0, s, ptrs + static_cast<int64_t>(g0) * n, n, sel, beta, tab);
      return hipGetLastError();
    });
  }
}

}  // namespace

int table_width(int n) { return n <= 12 ? 4 : (n <= 19 ? 2 : 1); }

int64_t table_tiles(const int64_t* dims, int K, int n) {
  const int w = table_width(n);
  int64_t t = 0;
  for (int s = 0; s < K; ++s) {
    const int64_t c = direct_chunk(dims[s], w);
    t += (dims[s] + c - 1) / c;
  }
  return t;
}

hipError_t enqueue_distances_table(const float* const* ptrs, int n, const int64_t* dims, int K,
                                   double* partial, int64_t tiles, hipStream_t s) {
  return dist_seg_dispatch<2>(n, ptrs, dims, K, partial, tiles, s);
}

hipError_t enqueue_mean_rows_table(const float* const* ptrs, int n, const int64_t* dims,
                                   float* const* outs, int K, const int32_t* rows, int k,
                                   hipStream_t s) {
  return for_each_launch(dims, outs, K, kAggSpan, [&](int g0, const SegTable& tab,
                                                        int64_t total) {
    if (rows)
      launch("mean_rows_seg", k_mean_rows_seg<4, true>, dim3(static_cast<unsigned>(total)),
             dim3(kBlock), 0, s, ptrs + static_cast<int64_t>(g0) * n, n, rows, k, tab);
    else
      launch("mean_rows_seg", k_mean_rows_seg<4, false>, dim3(static_cast<unsigned>(total)),
             dim3(kBlock), 0, s, ptrs + static_cast<int64_t>(g0) * n, n, rows, k, tab);
    return hipGetLastError();
  });
}

hipError_t enqueue_median_table(const float* const* ptrs, int n, const int64_t* dims,
                                float* const* outs, int K, hipStream_t s) {
  return median_seg_dispatch<1>(n, ptrs, dims, outs, K, s);
}

hipError_t enqueue_bulyan_table(const float* const* ptrs, int n, int f, const int64_t* dims,
                                float* const* outs, int K, const int32_t* sel, hipStream_t s) {
  const int theta = n - 2 * f;
  return bulyan_seg_dispatch<1>(theta, theta - 2 * f, ptrs, n, sel, dims, outs, K, s);
}

}  // namespace garfield
