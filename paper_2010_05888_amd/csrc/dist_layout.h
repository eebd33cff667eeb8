// How the distance step's per-entry sums map to D[i][j]. Shared by the
// kernels that consume distances (selection, MDA search, the D writer).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "internal.h"

namespace garfield {

// The result of the distance step: one fp64 sum per entry.
//  * direct engine: entry p = pair (i < j), row-major over i, holds D[i][j];
//  * Gram engine: entry q*256 + r*16 + c holds G[16*b1 + r][16*b2 + c] for the
//    q-th block pair (b1 <= b2) of the upper block triangle, G = Y Y^T;
//  * no engine (n < 2 or d == 0): D is all zeros;
//  * matrix: sums is the full n x n fp64 matrix D, row-major.
// Folded (direct engine with at most kFoldTiles tiles): sums is not formed;
// partial[entry * tiles + tile] holds the tiles' partial sums, and load_dist
// adds them exactly as the tile-sum kernel would (only load_dist reads this
// form).
struct DistSums {
  const double* sums;
  int engine;
  int n;
  const double* partial = nullptr;
  int64_t tiles = 0;
};

__device__ __forceinline__ int direct_entry(int n, int i, int j) {  // i < j
  return i * (2 * n - i - 1) / 2 + (j - i - 1);
}

__device__ __forceinline__ int gram_entry(int nb, int i, int j) {  // i <= j
  const int b1 = i >> 4, b2 = j >> 4;
  const int q = b1 * nb - b1 * (b1 - 1) / 2 + (b2 - b1);
  return q * 256 + (i & 15) * 16 + (j & 15);
}

// D[i][j] (symmetric, zero diagonal). The Gram form is evaluated in fp64 and
// clamped at 0; identical rows give exactly 0 because their G entries agree.
__device__ __forceinline__ double dist_entry(const DistSums& ds, int i, int j) {
  if (i == j || ds.engine == kEngineNone) return 0.0;
  if (ds.engine == kEngineMatrix) return ds.sums[i * ds.n + j];
  const int a = i < j ? i : j, b = i < j ? j : i;
  if (ds.engine == kEngineDirect) return ds.sums[direct_entry(ds.n, a, b)];
  const int nb = (ds.n + 15) / 16;
  const double v = (ds.sums[gram_entry(nb, a, a)] + ds.sums[gram_entry(nb, b, b)]) -
                   2.0 * ds.sums[gram_entry(nb, a, b)];
  return v > 0.0 ? v : 0.0;
}

// D into a block-shared n x n array (all threads of the block take part). For
// the Gram engine the diagonal G_ii is staged first, so that every entry then
// takes one load; D[i][j] is formed exactly as dist_entry forms it.
__device__ __forceinline__ void load_dist(const DistSums& ds, double* D) {
  const int n = ds.n;
  if (ds.partial) {
    // Entry e is the sum of tiles t = 0 .. tiles-1 in the tile-sum kernel's
    // order: slot u (< 256) holds tile u, then slots u and u + h are added for
    // h = 128, 64, ..., 1. Lane l of a wave holds slots l, l+64, l+128, l+192
    // and adds them as the levels 128 and 64 do; the xor butterfly from 32
    // down to 1 is the rest of the tree at lane 0 (for l < h, l ^ h = l + h).
    // A wave takes four entries at a time, all their loads issued first.
    __shared__ double esum[kDirectMaxNLimit * (kDirectMaxNLimit - 1) / 2];
    const int P = n * (n - 1) / 2;
    const int lane = threadIdx.x & 63, waves = blockDim.x >> 6;
    const int64_t t = ds.tiles;
    for (int e0 = threadIdx.x >> 6; e0 < P; e0 += 4 * waves) {
      double v[4] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int e = e0 + k * waves;  // wave-uniform
        if (e < P) {
          const double* row = ds.partial + static_cast<int64_t>(e) * t;
          const double s0 = lane < t ? row[lane] : 0.0;
          const double s1 = lane + 64 < t ? row[lane + 64] : 0.0;
          const double s2 = lane + 128 < t ? row[lane + 128] : 0.0;
          const double s3 = lane + 192 < t ? row[lane + 192] : 0.0;
          v[k] = (s0 + s2) + (s1 + s3);
        }
      }
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const int e = e0 + k * waves;
        if (e < P) {
#pragma unroll
          for (int m = 32; m > 0; m >>= 1) v[k] += __shfl_xor(v[k], m, 64);
          if (lane == 0) esum[e] = v[k];
        }
      }
    }
    __syncthreads();
    for (int idx = threadIdx.x; idx < n * n; idx += blockDim.x) {
      const int i = idx / n, j = idx % n;
      D[idx] = i == j ? 0.0 : esum[direct_entry(n, i < j ? i : j, i < j ? j : i)];
    }
  } else if (ds.engine == kEngineGram) {
    __shared__ double diag[kNmax];
    const int nb = (n + 15) / 16;
    if (static_cast<int>(threadIdx.x) < n) diag[threadIdx.x] = ds.sums[gram_entry(nb, threadIdx.x, threadIdx.x)];
    __syncthreads();
#pragma unroll 4
    for (int idx = threadIdx.x; idx < n * n; idx += blockDim.x) {
      const int i = idx / n, j = idx % n;
      const int a = i < j ? i : j, b = i < j ? j : i;
      const double v = (diag[a] + diag[b]) - 2.0 * ds.sums[gram_entry(nb, a, b)];
      D[idx] = (i == j) ? 0.0 : (v > 0.0 ? v : 0.0);
    }
  } else {
#pragma unroll 4
    for (int idx = threadIdx.x; idx < n * n; idx += blockDim.x) D[idx] = dist_entry(ds, idx / n, idx % n);
  }
  __syncthreads();
}

}  // namespace garfield
