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
// each summed in ascending thread order), whatever the pair. The sums are
// stored by lanes 0..31 of wave 0; COHERENT: as device-coherent (agent-scope
// atomic) stores, for a reader in another workgroup of the same launch.
template <int P, bool COHERENT = false>
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
      if constexpr (COHERENT)
        __hip_atomic_store(out + (base + t) * stride, a, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
      else
        out[(base + t) * stride] = a;
    }
    __syncthreads();
  }
}

// Column sums for the mean of a large selection (dist.hip's column-sum
// variant): colsum[c] is the fp64 sum of the N rows at coordinate c, in row
// order, when that sum and every sum of a subset of the rows is exact, else
// NaN. Exactness is decided from the exponents: finite fp32 values whose
// exponent fields lie in [emin, emax] (subnormals counted as 1) are integer
// multiples of 2^(emin - 150) below 2^(emax - 126) in magnitude, so any sum of
// at most 64 of them is such a multiple below 2^(emax - 120), which takes at
// most emax - emin + 30 bits: exact in fp64 when emax - emin <= 23. hi is the
// largest |bits| seen, lo1 the smallest |bits| - 1 (zeros wrap to 2^32 - 1
// and drop out).
struct ColSum {
  double s = 0.0;
  uint32_t hi = 0, lo1 = 0xffffffffu;
  __device__ __forceinline__ void add(float v) {
    const uint32_t b = __float_as_uint(v) & 0x7fffffffu;
    hi = b > hi ? b : hi;
    lo1 = (b - 1u) < lo1 ? (b - 1u) : lo1;
    s += static_cast<double>(v);
  }
  __device__ __forceinline__ double value() const {
    const int emax = static_cast<int>(hi >> 23);
    int emin = lo1 == 0xffffffffu ? emax : static_cast<int>((lo1 + 1u) >> 23);
    emin = emin < 1 ? 1 : emin;
    return (emax < 255 && emax - emin <= 23) ? s : __builtin_nan("");
  }
};

// The W coordinates c .. c+W-1 (c < end) of rows 0..N-1 into v; coordinates
// at or beyond end read as 0.
template <int N, int W, class Src>
__device__ __forceinline__ void direct_load(const Src& src, int64_t c, int64_t end,
                                            float (&v)[N][W]) {
  if (c + W <= end) {
#pragma unroll
    for (int i = 0; i < N; ++i) load_w<W>(src.row(i) + c, v[i]);
  } else {
#pragma unroll
    for (int i = 0; i < N; ++i) load_w_tail<W>(src.row(i) + c, end - c, v[i]);
  }
}

// acc[p] += (v[i][e] - v[j][e])^2 for every pair p = (i < j), row-major over
// i, coordinate by coordinate.
template <int N, int W>
__device__ __forceinline__ void direct_add(const float (&v)[N][W], float* acc) {
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

// The column sums (ColSum) of the W coordinates c .. c+W-1 (those before
// end) of the N rows in v, written to colsum.
template <int N, int W>
__device__ __forceinline__ void direct_colsum(const float (&v)[N][W], int64_t c, int64_t end,
                                              double* __restrict__ colsum) {
  double o[W];
#pragma unroll
  for (int e = 0; e < W; ++e) {
    ColSum cs;
#pragma unroll
    for (int i = 0; i < N; ++i) cs.add(v[i][e]);
    o[e] = cs.value();
  }
  // ordinary (L2-allocating) stores, two doubles at a time: the lanes' halves
  // of each cache line meet in L2 before it goes to HBM
  if constexpr (W >= 2) {
    if (c + W <= end) {
#pragma unroll
      for (int e = 0; e < W; e += 2) {
        d2 t;
        t.x = o[e];
        t.y = o[e + 1];
        *reinterpret_cast<d2*>(colsum + c + e) = t;
      }
      return;
    }
  }
#pragma unroll
  for (int e = 0; e < W; ++e)
    if (c + e < end) colsum[c + e] = o[e];
}

// Lane t takes W consecutive coordinates every kBlock * W in [start, end) of
// rows 0..N-1 of `src`, adding (x_i - x_j)^2 for every pair into acc (pairs
// in row-major order over i < j). With SUM, it also writes the column sums
// (ColSum) of its coordinates to colsum. The passes that lie wholly before
// `end` for every lane of the block are software-pipelined: the next pass's
// loads are issued before this pass's arithmetic, so the rows stream while
// the VALU works; the sums are formed in the same order either way.
template <int N, int W, bool SUM = false, class Src>
__device__ __forceinline__ void direct_accumulate(const Src& src, int64_t start, int64_t end,
                                                  float* acc, double* __restrict__ colsum = nullptr) {
  constexpr int64_t kStride = static_cast<int64_t>(kBlock) * W;
  const int64_t off = static_cast<int64_t>(threadIdx.x) * W;
  const int64_t full = end > start ? (end - start) / kStride : 0;  // block-uniform
  int64_t base = start;
  if (full > 0) {
    float v[N][W];
#pragma unroll
    for (int i = 0; i < N; ++i) load_w<W>(src.row(i) + base + off, v[i]);
    for (int64_t p = 1; p < full; ++p) {
      float nv[N][W];
#pragma unroll
      for (int i = 0; i < N; ++i) load_w<W>(src.row(i) + base + kStride + off, nv[i]);
      direct_add<N, W>(v, acc);
      if constexpr (SUM) direct_colsum<N, W>(v, base + off, end, colsum);
      base += kStride;
#pragma unroll
      for (int i = 0; i < N; ++i)
#pragma unroll
        for (int e = 0; e < W; ++e) v[i][e] = nv[i][e];
    }
    direct_add<N, W>(v, acc);
    if constexpr (SUM) direct_colsum<N, W>(v, base + off, end, colsum);
    base += kStride;
  }
  const int64_t c = base + off;  // the partial pass at the end, if any
  if (c < end) {
    float v[N][W];
    direct_load<N, W>(src, c, end, v);
    direct_add<N, W>(v, acc);
    if constexpr (SUM) direct_colsum<N, W>(v, c, end, colsum);
  }
}

}  // namespace garfield
