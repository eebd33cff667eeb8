// Contraction steps (decentralized learning, Section 5: each node repeatedly
// aggregates the vectors it receives from its peers). All N nodes' vectors are
// the rows of one N x d matrix x; node v's peers are peers[v*q .. v*q+q-1].
// One step writes every node's aggregate of its peers to row v of y. The
// selection kernel (k_peer_select) runs one workgroup per node on the
// distances of all N rows; the kernels below then aggregate every node in one
// launch. Mean and Median stage a 256-coordinate tile of all N rows in LDS
// (each input value read from HBM once, in 1 KB runs) and compute every
// node's output for that tile from it; Bulyan, bound by its per-node
// arithmetic rather than its loads, takes one workgroup per (tile, node), see
// node_grid. The per-coordinate arithmetic is the single-rule kernels' own.

#include "aggregate_body.h"
#include "internal.h"
#include "timing.h"

namespace garfield {

namespace {

// Workgroups of a step: every (tile, node) pair, mapped so that the nodes of one
// tile run back to back on one XCD. Workgroups are dispatched round-robin over
// the 8 XCDs; XCD x takes tiles x, x + 8, ..., and for each of them all nodes
// in turn, with ordinary (L2-allocating) loads, so the rows the nodes share
// come from that XCD's L2 after the first node read them. (Staging a tile of
// all rows in LDS and looping over the nodes in one workgroup was slower: the
// stage leaves one or two workgroups per CU.)
constexpr int kXcds = 8;

int64_t tiles_for(int64_t d, int w) {
  return (d + static_cast<int64_t>(kBlock) * w - 1) / (static_cast<int64_t>(kBlock) * w);
}

dim3 node_grid(int64_t tiles, int nodes) {
  const int64_t padded = (tiles + kXcds - 1) / kXcds * kXcds;
  return dim3(static_cast<unsigned>(padded * nodes));
}

// (tile, node) of this workgroup; tile may be past the last one (padding).
__device__ __forceinline__ void node_tile(int nodes, int64_t* tile, int* v) {
  const int64_t b = blockIdx.x;
  const int64_t j = b / kXcds;
  *tile = (j / nodes) * kXcds + b % kXcds;
  *v = static_cast<int>(j % nodes);
}

// LDS tile: coordinates c0 .. c0+255 of all n rows, row r at tile[r * 256].
// Wave w loads rows w, w + 4, ... with one 16-byte nontemporal load per lane
// (1 KB of a row per instruction), all of its rows before any store to LDS.
constexpr int kTileCoords = kBlock;
constexpr int kTileRowsPerWave = kNmax / 4;

__device__ __forceinline__ void stage_tile(const float* __restrict__ x, int n, int64_t d,
                                           int64_t c0, float* __restrict__ tile) {
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t c = c0 + 4 * lane;
  float v[kTileRowsPerWave][4];
#pragma unroll
  for (int u = 0; u < kTileRowsPerWave; ++u) {
    const int r = wave + 4 * u;  // wave-uniform
    if (r < n) {
      const float* p = x + static_cast<int64_t>(r) * d + c;
      if (c + 4 <= d) load_w<4>(p, v[u]); else load_w_tail<4>(p, d - c, v[u]);
    }
  }
#pragma unroll
  for (int u = 0; u < kTileRowsPerWave; ++u) {
    const int r = wave + 4 * u;
    if (r < n) {
      float* q = tile + r * kTileCoords + 4 * lane;
#pragma unroll
      for (int e = 0; e < 4; ++e) q[e] = v[u][e];
    }
  }
  __syncthreads();
}

// The nodes' row lists, as LDS offsets into the tile (row * 256), after the
// tile in dynamic LDS.
__device__ __forceinline__ int32_t* stage_offsets(const int32_t* __restrict__ rows, int count,
                                                  int n, float* tile) {
  int32_t* off = reinterpret_cast<int32_t*>(tile + n * kTileCoords);
  for (int i = threadIdx.x; i < count; i += kBlock)
    off[i] = static_cast<int32_t>(row_of(rows, i, n)) * kTileCoords;
  return off;
}

// Node v's output at coordinate c0 + t: the mean of its k rows (rows[v*k ..],
// fp64 sum in the order listed, one rounding), for every node; two nodes'
// sums at a time, so that two chains of additions are in flight.
__global__ __launch_bounds__(kBlock) void k_mean_nodes(const float* __restrict__ x, int n,
                                                       int64_t d, int nodes,
                                                       const int32_t* __restrict__ rows, int k,
                                                       float* __restrict__ y) {
  extern __shared__ float tile[];
  const int64_t c0 = static_cast<int64_t>(blockIdx.x) * kTileCoords;
  const int32_t* off = stage_offsets(rows, nodes * k, n, tile);
  stage_tile(x, n, d, c0, tile);  // ends with a barrier
  const int t = threadIdx.x;
  const int64_t c = c0 + t;
  if (c >= d) return;
  const double count = static_cast<double>(k);
  int v = 0;
  for (; v + 2 <= nodes; v += 2) {
    const int32_t* o0 = off + v * k;
    const int32_t* o1 = o0 + k;
    double a0 = 0.0, a1 = 0.0;
#pragma unroll 4
    for (int i = 0; i < k; ++i) {
      a0 += static_cast<double>(tile[o0[i] + t]);
      a1 += static_cast<double>(tile[o1[i] + t]);
    }
    __builtin_nontemporal_store(static_cast<float>(a0 / count), y + static_cast<int64_t>(v) * d + c);
    __builtin_nontemporal_store(static_cast<float>(a1 / count),
                                y + static_cast<int64_t>(v + 1) * d + c);
  }
  if (v < nodes) {
    const int32_t* o0 = off + v * k;
    double a0 = 0.0;
#pragma unroll 4
    for (int i = 0; i < k; ++i) a0 += static_cast<double>(tile[o0[i] + t]);
    __builtin_nontemporal_store(static_cast<float>(a0 / count), y + static_cast<int64_t>(v) * d + c);
  }
}

// Node v's output: the median of its K rows (the selection network of the
// single-rule median), for every node.
template <int K>
__global__ __launch_bounds__(kBlock) void k_median_nodes(const float* __restrict__ x, int n,
                                                         int64_t d, int nodes,
                                                         const int32_t* __restrict__ rows,
                                                         float* __restrict__ y) {
  using Net = MedianNet<K>;
  extern __shared__ float tile[];
  const int64_t c0 = static_cast<int64_t>(blockIdx.x) * kTileCoords;
  const int32_t* off = stage_offsets(rows, nodes * K, n, tile);
  stage_tile(x, n, d, c0, tile);  // ends with a barrier
  const int t = threadIdx.x;
  const int64_t c = c0 + t;
  if (c >= d) return;
  for (int v = 0; v < nodes; ++v) {
    const int32_t* ov = off + v * K;
    float a[K];
#pragma unroll
    for (int i = 0; i < K; ++i) a[i] = tile[ov[i] + t];
    Net::run(a);
    float o;
    if constexpr (K % 2 == 1) {
      o = a[Net::LO];
    } else {  // mean of the two middle values, exact in fp64, rounded once
      o = static_cast<float>((static_cast<double>(a[Net::LO]) + static_cast<double>(a[Net::HI])) *
                             0.5);
    }
    __builtin_nontemporal_store(o, y + static_cast<int64_t>(v) * d + c);
  }
}

unsigned tile_grid(int64_t d) {
  return static_cast<unsigned>((d + kTileCoords - 1) / kTileCoords);
}
// The tile and the nodes' row offsets (count entries).
size_t tile_bytes(int n, int count) {
  return static_cast<size_t>(n) * kTileCoords * sizeof(float) + count * sizeof(int32_t);
}

template <int T, int W>
__global__ __launch_bounds__(kBlock) void k_bulyan_nodes(const float* __restrict__ x, int n,
                                                         int64_t d, int nodes,
                                                         const int32_t* __restrict__ sel,
                                                         int beta, float* __restrict__ y) {
  __shared__ float sorted[T * kBlock];
  int64_t tile;
  int v;
  node_tile(nodes, &tile, &v);
  const int64_t c = (tile * kBlock + threadIdx.x) * W;
  if (c < d)
    bulyan_at<T, W, false>(MatrixRows{x, d}, d, ListedRows{sel + static_cast<int64_t>(v) * T, n},
                           beta, c, sorted + threadIdx.x, y + static_cast<int64_t>(v) * d);
}

// Bulyan's width as the single-rule kernel chooses it for float-aligned rows
// (the entry point requires those): the T x W values of a lane must fit the
// registers of two waves per SIMD.
template <int K>
hipError_t median_nodes_dispatch(int k, const float* x, int n, int64_t d, int nodes,
                                 const int32_t* rows, float* y, hipStream_t s) {
  if constexpr (K > kNmax) {
    return hipErrorInvalidValue;
  } else {
    if (k != K) return median_nodes_dispatch<K + 1>(k, x, n, d, nodes, rows, y, s);
    launch("median_nodes", k_median_nodes<K>, dim3(tile_grid(d)), dim3(kBlock),
           static_cast<uint32_t>(tile_bytes(n, nodes * K)), s, x, n, d, nodes, rows, y);
    return hipGetLastError();
  }
}

template <int T>
hipError_t bulyan_nodes_dispatch(int theta, int beta, const float* x, int n, int64_t d,
                                 int nodes, const int32_t* sel, float* y, hipStream_t s) {
  if constexpr (T > kNmax) {
    return hipErrorInvalidValue;
  } else {
    if (theta != T)
      return bulyan_nodes_dispatch<T + 1>(theta, beta, x, n, d, nodes, sel, y, s);
    constexpr int W = T <= 24 ? 4 : (T <= 48 ? 2 : 1);
    launch("bulyan_nodes", k_bulyan_nodes<T, W>, node_grid(tiles_for(d, W), nodes), dim3(kBlock),
           0, s, x, n, d, nodes, sel, beta, y);
    return hipGetLastError();
  }
}

}  // namespace

hipError_t enqueue_mean_nodes(const float* x, int n, int64_t d, int nodes, const int32_t* rows,
                              int k, float* y, hipStream_t s) {
  if (d == 0 || nodes == 0) return hipSuccess;
  launch("mean_nodes", k_mean_nodes, dim3(tile_grid(d)), dim3(kBlock),
         static_cast<uint32_t>(tile_bytes(n, nodes * k)), s, x, n, d, nodes, rows, k, y);
  return hipGetLastError();
}

hipError_t enqueue_median_nodes(const float* x, int n, int64_t d, int nodes, const int32_t* rows,
                                int k, float* y, hipStream_t s) {
  if (d == 0 || nodes == 0) return hipSuccess;
  return median_nodes_dispatch<1>(k, x, n, d, nodes, rows, y, s);
}

hipError_t enqueue_bulyan_nodes(const float* x, int n, int64_t d, int nodes, int q, int f,
                                const int32_t* sel, float* y, hipStream_t s) {
  if (d == 0 || nodes == 0) return hipSuccess;
  const int theta = q - 2 * f;
  return bulyan_nodes_dispatch<1>(theta, theta - 2 * f, x, n, d, nodes, sel, y, s);
}

}  // namespace garfield
