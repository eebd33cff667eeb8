// Contraction steps (decentralized learning, Section 5: each node repeatedly
// aggregates the vectors it receives from its peers). All N nodes' vectors are
// the rows of one N x d matrix x; node v's peers are peers[v*q .. v*q+q-1].
// One step writes every node's aggregate of its peers to row v of y. The
// selection kernel (k_peer_select) runs one workgroup per node on the
// distances of all N rows; the kernels below then aggregate every node in one
// launch (one workgroup per tile and node, see node_grid), with the
// per-coordinate code of the single-rule kernels (aggregate_body.h).

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

// Mean of node v's k rows (rows[v*k ..]), in the order listed.
template <int W>
__global__ __launch_bounds__(kBlock) void k_mean_nodes(const float* __restrict__ x, int n,
                                                       int64_t d, int nodes,
                                                       const int32_t* __restrict__ rows, int k,
                                                       float* __restrict__ y) {
  int64_t tile;
  int v;
  node_tile(nodes, &tile, &v);
  const int64_t c = (tile * kBlock + threadIdx.x) * W;
  if (c < d)
    mean_at<W, false>(MatrixRows{x, d}, n, d, rows + static_cast<int64_t>(v) * k, k, c,
                      y + static_cast<int64_t>(v) * d);
}

template <int K, int W>
__global__ __launch_bounds__(kBlock) void k_median_nodes(const float* __restrict__ x, int n,
                                                         int64_t d, int nodes,
                                                         const int32_t* __restrict__ rows,
                                                         float* __restrict__ y) {
  int64_t tile;
  int v;
  node_tile(nodes, &tile, &v);
  const int64_t c = (tile * kBlock + threadIdx.x) * W;
  if (c < d)
    median_at<K, W, false>(MatrixRows{x, d}, n, d, rows + static_cast<int64_t>(v) * K, c,
                           y + static_cast<int64_t>(v) * d);
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
    bulyan_at<T, W, false>(MatrixRows{x, d}, n, d, sel + static_cast<int64_t>(v) * T, beta, c,
                           sorted + threadIdx.x, y + static_cast<int64_t>(v) * d);
}

// Widths as the single-rule kernels choose them for float-aligned rows (the
// entry point requires those): the K (or T) x W values of a lane must fit the
// registers of two waves per SIMD.
template <int K>
hipError_t median_nodes_dispatch(int k, const float* x, int n, int64_t d, int nodes,
                                 const int32_t* rows, float* y, hipStream_t s) {
  if constexpr (K > kNmax) {
    return hipErrorInvalidValue;
  } else {
    if (k != K) return median_nodes_dispatch<K + 1>(k, x, n, d, nodes, rows, y, s);
    constexpr int W = K <= 52 ? 4 : 2;
    launch("median_nodes", k_median_nodes<K, W>, node_grid(tiles_for(d, W), nodes), dim3(kBlock),
           0, s, x, n, d, nodes, rows, y);
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
  launch("mean_nodes", k_mean_nodes<4>, node_grid(tiles_for(d, 4), nodes), dim3(kBlock), 0, s, x,
         n, d, nodes, rows, k, y);
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
