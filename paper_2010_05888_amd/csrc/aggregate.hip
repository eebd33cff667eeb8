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

#include "device_common.h"
#include "internal.h"
#include "timing.h"

namespace garfield {

#include "networks.inc"

namespace {

__device__ __forceinline__ int64_t row_of(const int32_t* __restrict__ rows, int t, int n) {
  if (!rows) return t;
  const int r = rows[t];
  return static_cast<int64_t>(r < 0 ? 0 : (r >= n ? n - 1 : r));
}

// ---------------------------------------------------------------------------
// fp64 sum of the k rows at coordinates c .. c+W-1, eight loads in flight at a
// time; FULL: all W coordinates exist (else the guarded tail loads).
template <int W, bool FULL>
__device__ __forceinline__ void sum_rows_at(const float* __restrict__ x, int n, int64_t d,
                                            const int32_t* __restrict__ rows, int k, int64_t c,
                                            double* acc) {
  int t = 0;
  for (; t + 8 <= k; t += 8) {
    float v[8][W];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const float* p = x + row_of(rows, t + u, n) * d + c;
      if constexpr (FULL) load_w<W>(p, v[u]); else load_w_tail<W>(p, d - c, v[u]);
    }
#pragma unroll
    for (int u = 0; u < 8; ++u)
#pragma unroll
      for (int e = 0; e < W; ++e) acc[e] += static_cast<double>(v[u][e]);
  }
  for (; t < k; ++t) {
    float v[W];
    const float* p = x + row_of(rows, t, n) * d + c;
    if constexpr (FULL) load_w<W>(p, v); else load_w_tail<W>(p, d - c, v);
#pragma unroll
    for (int e = 0; e < W; ++e) acc[e] += static_cast<double>(v[e]);
  }
}

template <int W>
__global__ __launch_bounds__(kBlock) void k_mean_rows(const float* __restrict__ x, int n,
                                                      int64_t d, const int32_t* __restrict__ rows,
                                                      int k, float* __restrict__ out) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock * W;
  const double count = static_cast<double>(k);
  for (int64_t c = (static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x) * W; c < d;
       c += stride) {
    double acc[W];
#pragma unroll
    for (int e = 0; e < W; ++e) acc[e] = 0.0;
    const bool full = c + W <= d;
    if (full) sum_rows_at<W, true>(x, n, d, rows, k, c, acc);
    else sum_rows_at<W, false>(x, n, d, rows, k, c, acc);
    float o[W];
#pragma unroll
    for (int e = 0; e < W; ++e) o[e] = static_cast<float>(acc[e] / count);
    if (full) {
      store_w<W>(out + c, o);
    } else {
      for (int e = 0; e < W && c + e < d; ++e) out[c + e] = o[e];
    }
  }
}

// ---------------------------------------------------------------------------
// Every lane loads W consecutive coordinates of each of the K rows: 16-byte
// loads (W = 4) stream a K-row gather far faster than 8- or 4-byte ones, so
// W = 4 is kept up to K = kMedianX4MaxK, where the K x 4 values still fit the
// registers of two waves per SIMD.
constexpr int kMedianX4MaxK = 52;

template <int K, int W>
__global__ __launch_bounds__(kBlock) void k_median(const float* __restrict__ x, int n, int64_t d,
                                                   const int32_t* __restrict__ rows,
                                                   float* __restrict__ out) {
  using Net = MedianNet<K>;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock * W;
  for (int64_t c = (static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x) * W; c < d;
       c += stride) {
    float v[K][W];
    const bool full = c + W <= d;
    if (full) {  // all K loads back to back, then the network
#pragma unroll
      for (int t = 0; t < K; ++t) load_w<W>(x + row_of(rows, t, n) * d + c, v[t]);
    } else {
#pragma unroll
      for (int t = 0; t < K; ++t) load_w_tail<W>(x + row_of(rows, t, n) * d + c, d - c, v[t]);
    }
    float o[W];
#pragma unroll
    for (int e = 0; e < W; ++e) {
      float a[K];
#pragma unroll
      for (int t = 0; t < K; ++t) a[t] = v[t][e];
      Net::run(a);
      if constexpr (K % 2 == 1) {
        o[e] = a[Net::LO];
      } else {  // mean of the two middle values, exact in fp64, rounded once
        o[e] = static_cast<float>((static_cast<double>(a[Net::LO]) +
                                   static_cast<double>(a[Net::HI])) * 0.5);
      }
    }
    if (full) {
      store_w<W>(out + c, o);
    } else {
      for (int e = 0; e < W && c + e < d; ++e) out[c + e] = o[e];
    }
  }
}

// ---------------------------------------------------------------------------
// Bulyan aggregation for theta = T selected rows, beta = T - 2f closest.
//
// With s[0..T-1] sorted: odd T has the median s[c], c = (T-1)/2, always kept,
// and K = beta-1 more to take; even T has med = (s[c-1]+s[c])/2, c = T/2, and
// K = beta to take. Left candidates L_a = s[c-a] (a = 1, 2, ...) and right
// candidates R_b (s[c+b] for odd T, s[c-1+b] for even T) are each ordered by
// increasing key, so the K taken are the first K of their merge: L_a is taken
// iff key(L_a) < key(R_{K+1-a}) (a missing R counts as +inf). The number of
// left values taken is the count of such a.
template <int T, int W>
__global__ __launch_bounds__(kBlock) void k_bulyan_agg(const float* __restrict__ x, int n,
                                                       int64_t d, const int32_t* __restrict__ sel,
                                                       int beta, float* __restrict__ out) {
  using Net = SortNet<T>;
  __shared__ float sorted[T * kBlock];
  float* col = sorted + threadIdx.x;  // column of this thread: col[r * kBlock]
  constexpr bool kOdd = (T % 2) == 1;
  constexpr int c = kOdd ? (T - 1) / 2 : T / 2;
  constexpr int n_left = c;                          // L_a exists for a <= n_left
  constexpr int n_right = kOdd ? T - 1 - c : T - c;  // R_b exists for b <= n_right
  const int K = kOdd ? beta - 1 : beta;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kBlock * W;
  for (int64_t cc = (static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x) * W; cc < d;
       cc += stride) {
    float v[T][W];
    const bool full = cc + W <= d;
    if (full) {
#pragma unroll
      for (int t = 0; t < T; ++t) load_w<W>(x + row_of(sel, t, n) * d + cc, v[t]);
    } else {
#pragma unroll
      for (int t = 0; t < T; ++t) load_w_tail<W>(x + row_of(sel, t, n) * d + cc, d - cc, v[t]);
    }
    float o[W];
#pragma unroll
    for (int e = 0; e < W; ++e) {
      float a[T];
#pragma unroll
      for (int t = 0; t < T; ++t) a[t] = v[t][e];
      Net::run(a);
#pragma unroll
      for (int r = 0; r < T; ++r) col[r * kBlock] = a[Net::reg(r)];
      const double med = kOdd ? static_cast<double>(col[c * kBlock])
                              : (static_cast<double>(col[(c - 1) * kBlock]) +
                                 static_cast<double>(col[c * kBlock])) * 0.5;
      int a_taken = 0;
      for (int i = 1; i <= K; ++i) {
        if (i > n_left) break;
        const int b = K + 1 - i;
        bool take = true;
        if (b <= n_right) {
          const float lv = col[(c - i) * kBlock];
          const float rv = col[(kOdd ? c + b : c - 1 + b) * kBlock];
          const double dl = med - static_cast<double>(lv);
          const double dr = static_cast<double>(rv) - med;
          take = (dl < dr) || (dl == dr && lv < rv);
        }
        if (!take) break;
        a_taken = i;
      }
      const int lo = c - a_taken;
      const int hi = lo + beta - 1;  // inclusive
      double sum = 0.0;
      for (int r = lo; r <= hi; ++r) sum += static_cast<double>(col[r * kBlock]);
      o[e] = static_cast<float>(sum / static_cast<double>(beta));
    }
    if (full) {
      store_w<W>(out + cc, o);
    } else {
      for (int e = 0; e < W && cc + e < d; ++e) out[cc + e] = o[e];
    }
  }
}

// ---------------------------------------------------------------------------
// One pass: a workgroup per kBlock items, so every lane handles one item (the
// grid-stride loops in the kernels only matter beyond 2^31 - 1 workgroups).
// A single pass streams measurably faster than a capped grid looping over d.
int grid_for(int64_t items) {
  int64_t blocks = (items + kBlock - 1) / kBlock;
  if (blocks > 0x7fffffff) blocks = 0x7fffffff;
  if (blocks < 1) blocks = 1;
  return static_cast<int>(blocks);
}

template <int W>
hipError_t launch_mean(const float* x, int n, int64_t d, const int32_t* rows, int k, float* out,
                       hipStream_t s) {
  launch("mean_rows", k_mean_rows<W>, dim3(grid_for((d + W - 1) / W)), dim3(kBlock), 0, s, x, n,
    d, rows, k, out);
  return hipGetLastError();
}

template <int K, int W>
hipError_t launch_median_kw(const float* x, int n, int64_t d, const int32_t* rows, float* out,
                            hipStream_t s) {
  launch("median", k_median<K, W>, dim3(grid_for((d + W - 1) / W)), dim3(kBlock), 0, s, x, n,
    d, rows, out);
  return hipGetLastError();
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
  launch("bulyan_agg", k_bulyan_agg<T, W>, dim3(grid_for((d + W - 1) / W)), dim3(kBlock), 0, s,
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
// out are float-aligned, whatever d (see f4u).
int stream_width(const float* x, const float* out) {
  return (vector_width(x) == 4 && vector_width(out) == 4) ? 4 : 1;
}

hipError_t enqueue_mean_rows(const float* x, int n, int64_t d, const int32_t* rows, int k,
                             float* out, hipStream_t s) {
  if (d == 0) return hipSuccess;
  const int w = stream_width(x, out);
  if (w == 4) return launch_mean<4>(x, n, d, rows, k, out, s);
  if (w == 2) return launch_mean<2>(x, n, d, rows, k, out, s);
  return launch_mean<1>(x, n, d, rows, k, out, s);
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

}  // namespace garfield
