// Pairwise squared distances D[i][j] = sum_c (x_ic - x_jc)^2 -- the O(n^2 d)
// step shared by Krum, Multi-Krum, MDA and Bulyan (Section 3.1 items 2-4;
// the paper's complexity discussion in Section 5.3 attributes the quadratic
// growth in n to it).
//
// The coordinates are cut into tiles of `chunk` consecutive coordinates, one
// workgroup per tile. Each tile writes fp64 partial sums; a second kernel sums
// the tiles in fixed-size segments and a third sums the segments, always in
// ascending order, so D is deterministic and depends only on (n, d), never on
// scheduling. Two engines:
//
//  * direct (n <= direct_max_n(), default 20): every lane accumulates (x_i - x_j)^2 for all
//    n(n-1)/2 pairs in fp32 registers over its coordinates. No cancellation,
//    and identical rows give bit-identical rows of D.
//  * Gram (larger n): G = Y Y^T with Y = X - x_ref (a per-coordinate shift by
//    one input row, chosen robustly by a small probe), on fp32 MFMA
//    (v_mfma_f32_16x16x4_f32, 16-row blocks, upper block triangle only), then
//    D_ij = G_ii + G_jj - 2 G_ij in fp64. Shifting by a central row keeps the
//    cancellation in that difference to a small factor. Identical rows give
//    identical products in the same order, hence identical G and D rows and
//    an exact 0 between them.

#include "device_common.h"
#include "internal.h"
#include "timing.h"

namespace garfield {

namespace {

// ---------------------------------------------------------------------------
// Block-wide reduction of P per-thread fp32 accumulators into P fp64 sums,
// through LDS in chunks of 32 columns (33-float row stride: conflict-free).
// Every sum is formed in the same order (eight fixed groups of 32 threads,
// each summed in ascending thread order), whatever the pair.
template <int P>
__device__ __forceinline__ void block_reduce_pairs(const float* acc, double* __restrict__ out) {
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
      out[base + t] = a;
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// Direct engine. Tile = `chunk` coordinates (a multiple of kBlock * W); lane t
// takes W consecutive coordinates every kBlock * W.
template <int N, int W>
__global__ __launch_bounds__(kBlock) void k_dist_direct(const float* __restrict__ x, int64_t d,
                                                         int64_t chunk,
                                                         double* __restrict__ partial) {
  constexpr int P = N * (N - 1) / 2;
  float acc[P];
#pragma unroll
  for (int p = 0; p < P; ++p) acc[p] = 0.0f;
  const int64_t start = static_cast<int64_t>(blockIdx.x) * chunk;
  const int64_t end = (start + chunk < d) ? start + chunk : d;
  for (int64_t c = start + static_cast<int64_t>(threadIdx.x) * W; c < end; c += kBlock * W) {
    float v[N][W];
    if (c + W <= end) {
#pragma unroll
      for (int i = 0; i < N; ++i) load_w<W>(x + static_cast<int64_t>(i) * d + c, v[i]);
    } else {
#pragma unroll
      for (int i = 0; i < N; ++i) load_w_tail<W>(x + static_cast<int64_t>(i) * d + c, end - c, v[i]);
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
  block_reduce_pairs<P>(acc, partial + static_cast<int64_t>(blockIdx.x) * P);
}

// ---------------------------------------------------------------------------
// Gram engine, step 1: probe. Block i sums (x_i - x_j)^2 over a sample of
// kProbeRuns runs of kBlock consecutive coordinates spread over d (all
// coordinates when d is small) for every j.
__global__ __launch_bounds__(kBlock) void k_probe(const float* __restrict__ x, int n, int64_t d,
                                                  float* __restrict__ probe) {
  __shared__ float red[kBlock];
  const int i = blockIdx.x;
  float acc[kNmax];
#pragma unroll
  for (int j = 0; j < kNmax; ++j) acc[j] = 0.0f;
  const int64_t runs = (d <= static_cast<int64_t>(kProbeRuns) * kBlock) ? 1 : kProbeRuns;
  const int64_t stride = d / runs;
  const int64_t len = (runs == 1) ? d : kBlock;
  for (int64_t r = 0; r < runs; ++r) {
    for (int64_t o = threadIdx.x; o < len; o += kBlock) {
      const int64_t c = r * stride + o;
      const float xi = x[static_cast<int64_t>(i) * d + c];
#pragma unroll
      for (int j = 0; j < kNmax; ++j) {
        if (j < n) {
          const float t = xi - x[static_cast<int64_t>(j) * d + c];
          acc[j] = __builtin_fmaf(t, t, acc[j]);
        }
      }
    }
  }
  for (int j = 0; j < n; ++j) {
    float a = 0.0f;
#pragma unroll
    for (int j2 = 0; j2 < kNmax; ++j2)
      if (j2 == j) a = acc[j2];
    red[threadIdx.x] = a;
    __syncthreads();
    for (int s = kBlock / 2; s > 0; s >>= 1) {
      if (threadIdx.x < s) red[threadIdx.x] += red[threadIdx.x + s];
      __syncthreads();
    }
    if (threadIdx.x == 0) probe[i * n + j] = red[0];
    __syncthreads();
  }
}

// Gram engine, step 2: the reference row is the one whose sum of its
// ceil(n/2) smallest probe distances (self included, which is 0) is lowest:
// with an honest majority this is a central, honest row.
__global__ __launch_bounds__(64) void k_pick_ref(const float* __restrict__ probe, int n,
                                                 int32_t* __restrict__ ref) {
  __shared__ float score[kNmax];
  const int i = threadIdx.x;
  if (i < n) {
    const int h = (n + 1) / 2;
    float s = 0.0f;
    // sum of the h smallest entries of row i (selection by rank, ties by index)
    for (int j = 0; j < n; ++j) {
      const float v = probe[i * n + j];
      int rank = 0;
      for (int j2 = 0; j2 < n; ++j2) {
        const float w = probe[i * n + j2];
        rank += (w < v) || (w == v && j2 < j);
      }
      if (rank < h) s += v;
    }
    score[i] = s;
  }
  __syncthreads();
  if (i == 0) {
    int best = 0;
    for (int j = 1; j < n; ++j)
      if (score[j] < score[best]) best = j;
    *ref = best;
  }
}

// Gram engine, step 3: G partial sums per tile on MFMA.
//
// v_mfma_f32_16x16x4_f32 operand layout (wave64): lane l supplies
// A[l % 16][l / 16] and B[l / 16][l % 16]; the result element D[4*(l/16)+e][l%16]
// is component e of lane l's accumulator. For a Gram block both operands are
// 16 rows of Y at the same 4 coordinates, so one register per lane serves as
// A (rows of block b1) and as B (rows of block b2). Each lane owns 8
// coordinates per 32-coordinate step: c0 + 16h + 4g + e (g = l / 16, h in
// {0,1}, e in 0..3), i.e. two 64-byte runs per row; which coordinate feeds
// which k slot does not matter for a Gram matrix as long as A and B agree.
//
// Each wave handles its own quarter of the tile; fp32 accumulators are
// flushed into fp64 every 4 k-slices (16 products), which bounds the fp32
// accumulation error of every G entry to a few dozen ulps of the sum of its
// absolute products.
template <int NB, int W>
__global__ __launch_bounds__(kBlock) void k_dist_gram(const float* __restrict__ x, int n,
                                                       int64_t d, int64_t chunk,
                                                       const int32_t* __restrict__ ref_idx,
                                                       double* __restrict__ partial) {
  constexpr int NBP = NB * (NB + 1) / 2;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int g = lane >> 4;
  const int r = lane & 15;
  const int ref = *ref_idx;
  const float* __restrict__ xref = x + static_cast<int64_t>(ref) * d;
  const float* rowp[NB];
  bool valid[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const int row = 16 * b + r;
    valid[b] = row < n;
    rowp[b] = x + static_cast<int64_t>(valid[b] ? row : 0) * d;
  }
  f4 acc[NBP];
  double acc64[NBP][4];
#pragma unroll
  for (int q = 0; q < NBP; ++q) {
    acc[q] = f4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int e = 0; e < 4; ++e) acc64[q][e] = 0.0;
  }
  const int64_t tile_start = static_cast<int64_t>(blockIdx.x) * chunk;
  const int64_t tile_end = (tile_start + chunk < d) ? tile_start + chunk : d;
  const int64_t wchunk = chunk / 4;
  const int64_t w_start = tile_start + wave * wchunk;
  const int64_t w_end_raw = w_start + wchunk;
  const int64_t w_end = (w_end_raw < tile_end) ? w_end_raw : tile_end;
  for (int64_t c0 = w_start; c0 < w_end; c0 += 32) {
    float xv[NB][8];
    float rv[8];
    if (c0 + 32 <= w_end) {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int64_t c = c0 + 16 * h + 4 * g;
#pragma unroll
        for (int u = 0; u < 4; u += W) load_w<W>(xref + c + u, rv + 4 * h + u);
#pragma unroll
        for (int b = 0; b < NB; ++b) {
#pragma unroll
          for (int u = 0; u < 4; u += W) {
            if (valid[b]) {
              load_w<W>(rowp[b] + c + u, xv[b] + 4 * h + u);
            } else {
#pragma unroll
              for (int e = 0; e < W; ++e) xv[b][4 * h + u + e] = 0.0f;
            }
          }
        }
      }
    } else {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int64_t c = c0 + 16 * h + 4 * g;
        load_w_tail<4>(xref + c, w_end - c, rv + 4 * h);
#pragma unroll
        for (int b = 0; b < NB; ++b) {
          if (valid[b]) {
            load_w_tail<4>(rowp[b] + c, w_end - c, xv[b] + 4 * h);
          } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) xv[b][4 * h + e] = 0.0f;
          }
        }
      }
    }
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int s = 0; s < 8; ++s) xv[b][s] = valid[b] ? (xv[b][s] - rv[s]) : 0.0f;
#pragma unroll
    for (int half = 0; half < 2; ++half) {
#pragma unroll
      for (int s = 4 * half; s < 4 * half + 4; ++s) {
        int q = 0;
#pragma unroll
        for (int b1 = 0; b1 < NB; ++b1)
#pragma unroll
          for (int b2 = b1; b2 < NB; ++b2) {
            acc[q] = __builtin_amdgcn_mfma_f32_16x16x4f32(xv[b1][s], xv[b2][s], acc[q], 0, 0, 0);
            ++q;
          }
      }
      // Flush after every 4 k-slices: each fp32 accumulator then holds a sum
      // of at most 16 products before it is added into fp64.
#pragma unroll
      for (int q = 0; q < NBP; ++q) {
        acc64[q][0] += static_cast<double>(acc[q].x);
        acc64[q][1] += static_cast<double>(acc[q].y);
        acc64[q][2] += static_cast<double>(acc[q].z);
        acc64[q][3] += static_cast<double>(acc[q].w);
        acc[q] = f4{0.0f, 0.0f, 0.0f, 0.0f};
      }
    }
  }
  // Sum the four waves' blocks (in wave order) and write the tile's partials:
  // entry q*256 + row*16 + col holds G[16*b1 + row][16*b2 + col].
  __shared__ double red[4][256];
  double* __restrict__ out = partial + static_cast<int64_t>(blockIdx.x) * (NBP * 256);
#pragma unroll
  for (int q = 0; q < NBP; ++q) {
#pragma unroll
    for (int e = 0; e < 4; ++e) red[wave][(4 * g + e) * 16 + r] = acc64[q][e];
    __syncthreads();
    const int t = threadIdx.x;
    out[q * 256 + t] = ((red[0][t] + red[1][t]) + red[2][t]) + red[3][t];
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// Tiles -> segments: seg[s][p] = sum of partial[t][p] over the tiles of
// segment s, in ascending t.
__global__ __launch_bounds__(kBlock) void k_reduce_tiles(const double* __restrict__ partial,
                                                         int64_t tiles, int entries,
                                                         int64_t tiles_per_seg,
                                                         double* __restrict__ seg) {
  const int p = blockIdx.x * kBlock + threadIdx.x;
  const int s = blockIdx.y;
  if (p >= entries) return;
  const int64_t t0 = static_cast<int64_t>(s) * tiles_per_seg;
  const int64_t t1 = (t0 + tiles_per_seg < tiles) ? t0 + tiles_per_seg : tiles;
  double a = 0.0;
  for (int64_t t = t0; t < t1; ++t) a += partial[t * entries + p];
  seg[static_cast<int64_t>(s) * entries + p] = a;
}

__device__ __forceinline__ double sum_segments(const double* __restrict__ seg, int segs,
                                               int entries, int p) {
  double a = 0.0;
  for (int s = 0; s < segs; ++s) a += seg[static_cast<int64_t>(s) * entries + p];
  return a;
}

// Segments -> D (n x n fp64), direct engine: entry p enumerates i < j row-major.
__global__ __launch_bounds__(kBlock) void k_finalize_direct(const double* __restrict__ seg,
                                                            int segs, int n,
                                                            double* __restrict__ dist) {
  const int entries = n * (n - 1) / 2;
  for (int idx = threadIdx.x; idx < n * n; idx += kBlock) {
    const int i = idx / n, j = idx % n;
    double v = 0.0;
    if (i != j) {
      const int a = i < j ? i : j, b = i < j ? j : i;
      const int p = a * (2 * n - a - 1) / 2 + (b - a - 1);
      v = sum_segments(seg, segs, entries, p);
    }
    dist[idx] = v;
  }
}

// Segments -> D, Gram engine: G entries as laid out by k_dist_gram, then
// D_ij = G_ii + G_jj - 2 G_ij (clamped at 0), D_ii = 0.
__device__ __forceinline__ int gram_entry(int nb, int i, int j) {  // requires i <= j
  const int b1 = i >> 4, b2 = j >> 4;
  const int q = b1 * nb - b1 * (b1 - 1) / 2 + (b2 - b1);
  return q * 256 + (i & 15) * 16 + (j & 15);
}

__global__ __launch_bounds__(kBlock) void k_finalize_gram(const double* __restrict__ seg, int segs,
                                                          int n, int nb,
                                                          double* __restrict__ dist) {
  __shared__ double diag[kNmax];
  const int entries = nb * (nb + 1) / 2 * 256;
  for (int i = threadIdx.x; i < n; i += kBlock)
    diag[i] = sum_segments(seg, segs, entries, gram_entry(nb, i, i));
  __syncthreads();
  for (int idx = threadIdx.x; idx < n * n; idx += kBlock) {
    const int i = idx / n, j = idx % n;
    double v = 0.0;
    if (i != j) {
      const int a = i < j ? i : j, b = i < j ? j : i;
      const double gab = sum_segments(seg, segs, entries, gram_entry(nb, a, b));
      v = (diag[a] + diag[b]) - 2.0 * gab;
      v = v > 0.0 ? v : 0.0;
    }
    dist[idx] = v;
  }
}

__global__ void k_zero_f64(double* __restrict__ p, int count) {
  for (int idx = threadIdx.x; idx < count; idx += blockDim.x) p[idx] = 0.0;
}

// ---------------------------------------------------------------------------
template <int N, int W>
hipError_t launch_direct_nw(const float* x, const DistPlan& p, double* partial, hipStream_t s) {
  {
    TimedLaunch timed("dist_direct", s);
    hipLaunchKernelGGL((k_dist_direct<N, W>), dim3(static_cast<unsigned>(p.tiles)), dim3(kBlock), 0,
                       s, x, p.d, p.chunk, partial);
  }
  return hipGetLastError();
}

// Vector width the direct engine uses for n rows (register budget).
int direct_width_cap(int n) { return n <= 8 ? 4 : (n <= 16 ? 2 : 1); }

template <int N>
hipError_t launch_direct_n(const float* x, const DistPlan& p, double* partial, hipStream_t s) {
  if constexpr (N <= 8) {
    if (p.width == 4) return launch_direct_nw<N, 4>(x, p, partial, s);
  }
  if constexpr (N <= 16) {
    if (p.width >= 2) return launch_direct_nw<N, 2>(x, p, partial, s);
  }
  return launch_direct_nw<N, 1>(x, p, partial, s);
}

template <int N>
hipError_t launch_direct_dispatch(int n, const float* x, const DistPlan& p, double* partial,
                                  hipStream_t s) {
  if constexpr (N > kDirectMaxNLimit) {
    return hipErrorInvalidValue;
  } else {
    if (n == N) return launch_direct_n<N>(x, p, partial, s);
    return launch_direct_dispatch<N + 1>(n, x, p, partial, s);
  }
}

template <int NB, int W>
hipError_t launch_gram_nw(const float* x, const DistPlan& p, const int32_t* ref, double* partial,
                          hipStream_t s) {
  {
    TimedLaunch timed("dist_gram", s);
    hipLaunchKernelGGL((k_dist_gram<NB, W>), dim3(static_cast<unsigned>(p.tiles)), dim3(kBlock), 0,
                       s, x, p.n, p.d, p.chunk, ref, partial);
  }
  return hipGetLastError();
}

template <int NB>
hipError_t launch_gram_nb(const float* x, const DistPlan& p, const int32_t* ref, double* partial,
                          hipStream_t s) {
  if (p.width == 4) return launch_gram_nw<NB, 4>(x, p, ref, partial, s);
  if (p.width == 2) return launch_gram_nw<NB, 2>(x, p, ref, partial, s);
  return launch_gram_nw<NB, 1>(x, p, ref, partial, s);
}

size_t align256(size_t b) { return (b + 255) & ~static_cast<size_t>(255); }

int g_direct_max_n = 20;

}  // namespace

int direct_max_n() { return __atomic_load_n(&g_direct_max_n, __ATOMIC_RELAXED); }
void set_direct_max_n(int n) { __atomic_store_n(&g_direct_max_n, n, __ATOMIC_RELAXED); }

int load_width(const float* x, int64_t d) {
  const uintptr_t a = reinterpret_cast<uintptr_t>(x);
  if (d % 4 == 0 && a % 16 == 0) return 4;
  if (d % 2 == 0 && a % 8 == 0) return 2;
  return 1;
}

DistPlan plan_distances(int n, int64_t d, const float* x) {
  DistPlan p;
  p.n = n;
  p.d = d;
  if (n < 2 || d == 0) return p;  // D is all zeros
  p.width = load_width(x, d);
  if (n <= direct_max_n()) {
    p.engine = kEngineDirect;
    if (p.width > direct_width_cap(n)) p.width = direct_width_cap(n);
    // kDirectLaneCoords coordinates per lane per tile: each fp32 accumulator
    // sums at most that many squares before the tile is reduced in fp64.
    p.chunk = static_cast<int64_t>(kBlock) * kDirectLaneCoords;
    p.entries = n * (n - 1) / 2;
  } else {
    p.engine = kEngineGram;
    const int64_t step = 128 * 16;  // 4 waves x 32 coordinates x at least 16 steps
    int64_t chunk = (d + 1023) / 1024;
    chunk = (chunk + step - 1) / step * step;
    p.chunk = chunk;
    const int nb = (n + 15) / 16;
    p.entries = nb * (nb + 1) / 2 * 256;
  }
  p.tiles = (d + p.chunk - 1) / p.chunk;
  p.tiles_per_seg = (p.tiles + kMaxSegs - 1) / kMaxSegs;
  p.segs = static_cast<int>((p.tiles + p.tiles_per_seg - 1) / p.tiles_per_seg);
  return p;
}

size_t dist_workspace_bytes(const DistPlan& p) {
  size_t b = align256(static_cast<size_t>(p.n) * p.n * sizeof(double));
  if (p.engine != kEngineNone) {
    b += align256(static_cast<size_t>(p.tiles) * p.entries * sizeof(double));
    b += align256(static_cast<size_t>(p.segs) * p.entries * sizeof(double));
  }
  if (p.engine == kEngineGram) {
    b += align256(static_cast<size_t>(p.n) * p.n * sizeof(float));
    b += align256(sizeof(int32_t));
  }
  return b;
}

DistWorkspace carve_dist_workspace(const DistPlan& p, void* base) {
  DistWorkspace w;
  char* c = static_cast<char*>(base);
  w.dist = reinterpret_cast<double*>(c);
  c += align256(static_cast<size_t>(p.n) * p.n * sizeof(double));
  if (p.engine != kEngineNone) {
    w.partial = reinterpret_cast<double*>(c);
    c += align256(static_cast<size_t>(p.tiles) * p.entries * sizeof(double));
    w.seg = reinterpret_cast<double*>(c);
    c += align256(static_cast<size_t>(p.segs) * p.entries * sizeof(double));
  }
  if (p.engine == kEngineGram) {
    w.probe = reinterpret_cast<float*>(c);
    c += align256(static_cast<size_t>(p.n) * p.n * sizeof(float));
    w.ref = reinterpret_cast<int32_t*>(c);
  }
  return w;
}

hipError_t enqueue_reference(const float* x, const DistPlan& p, const DistWorkspace& ws,
                             hipStream_t s) {
  {
    TimedLaunch timed("probe", s);
    hipLaunchKernelGGL(k_probe, dim3(p.n), dim3(kBlock), 0, s, x, p.n, p.d, ws.probe);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  {
    TimedLaunch timed("pick_ref", s);
    hipLaunchKernelGGL(k_pick_ref, dim3(1), dim3(64), 0, s, ws.probe, p.n, ws.ref);
  }
  return hipGetLastError();
}

hipError_t enqueue_distances(const float* x, const DistPlan& p, const DistWorkspace& ws,
                             hipStream_t s) {
  hipError_t e = hipSuccess;
  if (p.engine == kEngineNone) {
    {
      TimedLaunch timed("zero", s);
      hipLaunchKernelGGL(k_zero_f64, dim3(1), dim3(kBlock), 0, s, ws.dist, p.n * p.n);
    }
    return hipGetLastError();
  }
  if (p.engine == kEngineDirect) {
    e = launch_direct_dispatch<2>(p.n, x, p, ws.partial, s);
  } else {
    if ((e = enqueue_reference(x, p, ws, s)) != hipSuccess) return e;
    const int nb = (p.n + 15) / 16;
    switch (nb) {
      case 1: e = launch_gram_nb<1>(x, p, ws.ref, ws.partial, s); break;
      case 2: e = launch_gram_nb<2>(x, p, ws.ref, ws.partial, s); break;
      case 3: e = launch_gram_nb<3>(x, p, ws.ref, ws.partial, s); break;
      case 4: e = launch_gram_nb<4>(x, p, ws.ref, ws.partial, s); break;
      default: return hipErrorInvalidValue;
    }
  }
  if (e != hipSuccess) return e;
  const dim3 grid((p.entries + kBlock - 1) / kBlock, p.segs);
  {
    TimedLaunch timed("reduce_tiles", s);
    hipLaunchKernelGGL(k_reduce_tiles, grid, dim3(kBlock), 0, s, ws.partial, p.tiles, p.entries,
                       p.tiles_per_seg, ws.seg);
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if (p.engine == kEngineDirect) {
    {
      TimedLaunch timed("finalize", s);
      hipLaunchKernelGGL(k_finalize_direct, dim3(1), dim3(kBlock), 0, s, ws.seg, p.segs, p.n,
                         ws.dist);
    }
  } else {
    {
      TimedLaunch timed("finalize", s);
      hipLaunchKernelGGL(k_finalize_gram, dim3(1), dim3(kBlock), 0, s, ws.seg, p.segs, p.n,
                         (p.n + 15) / 16, ws.dist);
    }
  }
  return hipGetLastError();
}

}  // namespace garfield
