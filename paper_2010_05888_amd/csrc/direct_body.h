// The direct distance engine's per-tile body, shared by the kernel over one
// row-major matrix (dist.hip) and the kernel over a table of segments
// (segtable.hip): per lane, fp32 sums of (x_i - x_j)^2 for every pair over
// its coordinates, then one block-wide reduction into fp64 partial sums.
#pragma once

#include "device_common.h"
#include "internal.h"
#include "rows.h"

namespace garfield {

// Block-wide reduction of P per-thread fp32 accumulators into P fp64 sums,
// through LDS in chunks of 32 columns (33-float row stride: conflict-free).
// Every sum is formed in the same order (eight fixed groups of 32 threads,
// each summed in ascending thread order), whatever the pair.
template <int P>
__device__ __forceinline__ void block_reduce_pairs(const float* acc, double* __restrict__ out,
                                                   int64_t stride) {
  __shared__ float cols[kBlock * 33];
  __shared__ double part[8][32];
  const int t = threadIdx.x;
#pragma unroll
  for (int base = 0; base < P; base += 32) {
#pragma unroll
    for (int q = 0; q < 32; ++q)
      if (base + q < P) cols[t * 33 + q] = acc[base + q];
    __syncthreads();
    const int q = t & 31, r = t >> 5;
    double s = 0.0;
    if (base + q < P) {
#pragma unroll 8
      for (int u = 0; u < 32; ++u) s += static_cast<double>(cols[(r * 32 + u) * 33 + q]);
    }
    part[r][q] = s;
    __syncthreads();
    if (t < 32 && base + t < P) {
      double a = part[0][t];
#pragma unroll
      for (int g = 1; g < 8; ++g) a += part[g][t];
      out[(base + t) * stride] = a;
    }
    __syncthreads();
  }
}

// Lane t takes W consecutive coordinates every kBlock * W in [start, end) of
// rows 0..N-1 of `src`, adding (x_i - x_j)^2 for every pair into acc (pairs
// in row-major order over i < j).
template <int N, int W, class Src>
__device__ __forceinline__ void direct_accumulate(const Src& src, int64_t start, int64_t end,
                                                  float* acc) {
  for (int64_t c = start + static_cast<int64_t>(threadIdx.x) * W; c < end; c += kBlock * W) {
    float v[N][W];
    if (c + W <= end) {
#pragma unroll
      for (int i = 0; i < N; ++i) load_w<W>(src.row(i) + c, v[i]);
    } else {
#pragma unroll
      for (int i = 0; i < N; ++i) load_w_tail<W>(src.row(i) + c, end - c, v[i]);
    }
#pragma unroll
    for (int e = 0; e < W; ++e) {
      int p = 0;
#pragma unroll
      for (int i = 0; i < N; ++i) {
#pragma unroll
        for (int j = i + 1; j < N; ++j) {
          const float t = v[i][e] - v[j][e];
          acc[p] = __builtin_fmaf(t, t, acc[p]);
          ++p;
        }
      }
    }
  }
}

}  // namespace garfield
