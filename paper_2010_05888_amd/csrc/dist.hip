// Pairwise squared distances D[i][j] = sum_c (x_ic - x_jc)^2 -- the O(n^2 d)
// step shared by Krum, Multi-Krum, MDA and Bulyan (Section 3.1 items 2-4;
// the paper's complexity discussion in Section 6.3 attributes the quadratic
// growth in n to it).
//
// Every workgroup of the distance kernel is a tile: the direct engine cuts the
// coordinates into tiles of `chunk` consecutive coordinates, the Gram engine
// gives workgroup b the 256-coordinate stages b, b + G, b + 2G, ... Each tile
// writes one fp64 partial sum per entry (entry-major: partial[entry * tiles +
// tile]); k_sum_tiles then adds the tiles of each entry in a fixed order, so D
// is deterministic and depends only on (n, d), never on scheduling. The
// consumers build D from the entry sums (dist_layout.h). Two engines:
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
#include "direct_body.h"
#include "dist_layout.h"
#include "internal.h"
#include "timing.h"

namespace garfield {

namespace {

// ---------------------------------------------------------------------------
// Direct engine (direct_body.h). Tile = `chunk` coordinates (a multiple of
// kBlock * W); lane t takes W consecutive coordinates every kBlock * W.
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
  direct_accumulate<N, W>(MatrixRows{x, d}, start, end, acc);
  block_reduce_pairs<P>(acc, partial + blockIdx.x, gridDim.x);
}

// The same step, also writing the exact column sums of the n rows (ColSum in
// direct_body.h) for the mean of a large selection.
template <int N, int W>
__global__ __launch_bounds__(kBlock) void k_dist_direct_sum(const float* __restrict__ x, int64_t d,
                                                             int64_t chunk,
                                                             double* __restrict__ partial,
                                                             double* __restrict__ colsum) {
  constexpr int P = N * (N - 1) / 2;
  float acc[P];
#pragma unroll
  for (int p = 0; p < P; ++p) acc[p] = 0.0f;
  const int64_t start = static_cast<int64_t>(blockIdx.x) * chunk;
  const int64_t end = (start + chunk < d) ? start + chunk : d;
  direct_accumulate<N, W, true>(MatrixRows{x, d}, start, end, acc, colsum);
  block_reduce_pairs<P>(acc, partial + blockIdx.x, gridDim.x);
}

// ---------------------------------------------------------------------------
// Gram engine, step 1: probe. The sample is kProbeRuns runs of kBlock
// consecutive coordinates spread evenly over d (all of d in one run when d is
// smaller than the sample). Workgroup (i, r) sums (x_i - x_j)^2 for every j
// over run r and writes row i of run r's probe matrix (kNmax x kNmax, fp64):
// one workgroup per row and run keeps the rows' scattered first touches in
// flight together rather than one run after another.
int probe_runs(int64_t d) {
  return d <= static_cast<int64_t>(kProbeRuns) * kBlock ? 1 : kProbeRuns;
}

template <class Src>
__global__ __launch_bounds__(kBlock) void k_probe(Src src, int n, int64_t d,
                                                  double* __restrict__ probe) {
  const int i = blockIdx.x, r = blockIdx.y;
  float acc[kNmax];
#pragma unroll
  for (int j = 0; j < kNmax; ++j) acc[j] = 0.0f;
  const int64_t runs = gridDim.y;
  const int64_t len = (runs == 1) ? d : kBlock;
  const int64_t first = r * (d / runs);
  for (int64_t o = threadIdx.x; o < len; o += kBlock) {
    const int64_t c = first + o;
    const float xi = src.row(i)[c];
#pragma unroll
    for (int j = 0; j < kNmax; ++j) {
      if (j < n) {
        const float t = xi - src.row(j)[c];
        acc[j] = __builtin_fmaf(t, t, acc[j]);
      }
    }
  }
  block_reduce_pairs<kNmax>(acc, probe + (static_cast<int64_t>(r) * kNmax + i) * kNmax, 1);
}

// Gram engine, step 2: the reference row is the one whose sum of its
// ceil(n/2) smallest probe distances (self included, which is 0) is lowest:
// with an honest majority this is a central, honest row. The probe distance
// of (i, j) is the sum of the runs' partial sums in run order (every thread
// issues all its loads before the first sum). Wave w of the 16 scores rows
// w, w + 16, ...: lane j ranks entry (i, j) in row i (ties by index) and the
// entries ranked below h are summed across the wave; wave 0 then takes the
// lowest (score, row).
constexpr int kPickThreads = 1024;

__global__ __launch_bounds__(kPickThreads) void k_pick_ref(const double* __restrict__ probe, int n,
                                                           int runs, int32_t* __restrict__ ref) {
  constexpr int kPer = kNmax * kNmax / kPickThreads;
  __shared__ double P[kNmax * kNmax];  // row stride kNmax; entries beyond n unused
  __shared__ double score[kNmax];
  double v[kPer];
#pragma unroll
  for (int k = 0; k < kPer; ++k) v[k] = 0.0;
  for (int r = 0; r < runs; ++r) {
    const double* q = probe + static_cast<int64_t>(r) * kNmax * kNmax;
    double t[kPer];
#pragma unroll
    for (int k = 0; k < kPer; ++k) t[k] = q[threadIdx.x + k * kPickThreads];
#pragma unroll
    for (int k = 0; k < kPer; ++k) v[k] += t[k];
  }
#pragma unroll
  for (int k = 0; k < kPer; ++k) P[threadIdx.x + k * kPickThreads] = v[k];
  __syncthreads();
  const int h = (n + 1) / 2;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  for (int i = wave; i < n; i += kPickThreads / 64) {
    const double* row = P + i * kNmax;
    const double x = lane < n ? row[lane] : 0.0;
    int rank = 0;
#pragma unroll 8
    for (int j2 = 0; j2 < n; ++j2) {
      const double w = row[j2];
      rank += (w < x) | ((w == x) & (j2 < lane));
    }
    const double s = wave_sum(lane < n && rank < h ? x : 0.0);
    if (lane == 0) score[i] = s;
  }
  __syncthreads();
  if (wave == 0) {
    const int best = wave_argmin_lane(lane < n ? score[lane] : __builtin_inf());
    if (lane == 0) *ref = best;
  }
}

// ---------------------------------------------------------------------------
// Gram engine, step 3: partial sums of G = Y Y^T, Y = X - x_ref, on fp32 MFMA
// (v_mfma_f32_16x16x4_f32), upper block triangle only.
//
// Streaming. A stage is the 16*NB rows (rows at or beyond n are not loaded;
// their Y rows are 0) times kGramStage = 256
// consecutive coordinates: 1 KB of every row, the shortest run that streams
// well from rows whose starts are not cache-line aligned (row i starts at
// i * d floats). Wave w loads rows w*4NB .. w*4NB + 4NB - 1 with one 16-byte
// load per lane per row (lane l: coordinates 4l .. 4l+3, so one instruction
// reads 1 KB of one row), writes them to the stage buffer in LDS, and issues
// the next stage's loads into the same registers before the stage is
// multiplied: a stage is in flight while the previous one is computed.
//
// Multiplying. The stage buffer holds Y (the reference row is subtracted as
// the stage is written). Wave w takes half h = w % 2 of the stage's
// coordinates (128) for the block pairs (b1 <= b2) of parity w / 2 (pairs q
// with q % 2 == w / 2; five each when NB = 4, so every wave issues the same
// number of MFMAs): per 16-coordinate group, lane (g = l/16, r = l%16) reads
// the 16-byte fragment of row 16b + r at coordinates 4g .. 4g+3 of each block
// b once (the A and B operands of four consecutive MFMA k-steps). Each pair's
// MFMAs over two groups start from zero and their fp32 result (32 products)
// is added into fp64, so every fp32 accumulation spans 32 products whatever d
// is. (The conversions and fp64 additions do not overlap the MFMAs on this
// hardware: one addition per 32 products instead of per 16 saves about a
// fifth of the multiply time.)
//
// Partials. The two halves' fp64 sums of each pair are added (half 0 first)
// and written as this workgroup's partials; workgroup b takes stages b, b + G, ... (G = grid
// size), so at any time the grid streams one compact window of every row.
constexpr int kGramStage = 256;               // coordinates per stage
constexpr int kGramPitch = kGramStage + 4;    // floats per LDS row (bank spread)

template <int NB>
struct GramShape {
  static constexpr int ROWS = 16 * NB;
  static constexpr int NBP = NB * (NB + 1) / 2;   // block pairs b1 <= b2
  static constexpr int RPW = ROWS / 4;            // rows loaded per wave
  static constexpr int PPW = (NBP + 1) / 2;       // pairs per wave (one parity)
};

__host__ __device__ constexpr int pair_b1(int nb, int q) {
  int b1 = 0;
  while (q >= nb - b1) {
    q -= nb - b1;
    ++b1;
  }
  return b1;
}
__host__ __device__ constexpr int pair_b2(int nb, int q) {
  int b1 = 0;
  while (q >= nb - b1) {
    q -= nb - b1;
    ++b1;
  }
  return b1 + q;
}

// LDS-only barrier: waits for this wave's LDS operations, then for every
// wave, and leaves vector-memory loads in flight (a __syncthreads() would also
// wait for those).
__device__ __forceinline__ void lds_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(0xC07F);  // lgkmcnt(0); vmcnt and expcnt unconstrained
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Issue the loads of the stage at c0: this wave's rows into v, the reference
// row into vr (coordinates at or beyond d read as 0 when the stage is the
// partial last one).
template <int NB, bool PAD, bool FULL, class Src>
__device__ __forceinline__ void gram_issue(const Src& src, int n, int64_t d, int ref, int wave,
                                           int lane, int64_t c0, f4* v, f4& vr) {
  using S = GramShape<NB>;
  const int64_t c = c0 + 4 * lane;
  auto load = [&](int row, f4& out) {
    const float* p = src.row(row) + c;
    float t[4];
    if constexpr (FULL) {
      load_w<4>(p, t);
    } else {
      if (c + 4 <= d) load_w<4>(p, t); else load_w_tail<4>(p, d - c, t);
    }
    out = f4{t[0], t[1], t[2], t[3]};
  };
#pragma unroll
  for (int i = 0; i < S::RPW; ++i) {
    const int row = wave * S::RPW + i;  // wave-uniform
    if (!PAD || row < n) load(row, v[i]);
  }
  load(ref, vr);
}

// Y = X - x_ref for this wave's rows into the stage buffer (rows at or beyond
// n are 0).
template <int NB, bool PAD>
__device__ __forceinline__ void gram_put(float* __restrict__ buf, int n, int wave, int lane,
                                         const f4* v, const f4& vr) {
  using S = GramShape<NB>;
#pragma unroll
  for (int i = 0; i < S::RPW; ++i) {
    const int row = wave * S::RPW + i;  // wave-uniform
    f4 t = v[i] - vr;
    if (PAD && row >= n) t = f4{0.0f, 0.0f, 0.0f, 0.0f};
    *reinterpret_cast<f4*>(buf + row * kGramPitch + 4 * lane) = t;
  }
}

// Pairs I, I + 1, ... of this wave (pair q = 2I + PH) over two consecutive
// 16-coordinate groups (fragments y0, y1): per pair a chain of eight MFMAs (32
// products) from zero, then one addition into fp64. Two pairs at a time, their
// chains interleaved, so that no MFMA waits on the one issued just before it.
// A template recursion, so that every pair's blocks are compile-time
// constants (the fragments stay in fixed registers).
template <int NB, int Q>
__device__ __forceinline__ void gram_flush(const f4& acc, double* acc64) {
  (void)Q;
  acc64[0] += static_cast<double>(acc.x);
  acc64[1] += static_cast<double>(acc.y);
  acc64[2] += static_cast<double>(acc.z);
  acc64[3] += static_cast<double>(acc.w);
}

template <int NB, int PH, int I>
__device__ __forceinline__ void gram_pairs(const f4* y0, const f4* y1, double (*acc64)[4]) {
  using S = GramShape<NB>;
  constexpr int q = 2 * I + PH;
  constexpr int q2 = 2 * (I + 1) + PH;
  const f4 zero = f4{0.0f, 0.0f, 0.0f, 0.0f};
  if constexpr (I + 1 < S::PPW && q2 < S::NBP) {
    constexpr int a1 = pair_b1(NB, q), a2 = pair_b2(NB, q);
    constexpr int c1 = pair_b1(NB, q2), c2 = pair_b2(NB, q2);
    f4 u = __builtin_amdgcn_mfma_f32_16x16x4f32(y0[a1].x, y0[a2].x, zero, 0, 0, 0);
    f4 w = __builtin_amdgcn_mfma_f32_16x16x4f32(y0[c1].x, y0[c2].x, zero, 0, 0, 0);
    u = __builtin_amdgcn_mfma_f32_16x16x4f32(y0[a1].y, y0[a2].y, u, 0, 0, 0);
    w = __builtin_amdgcn_mfma_f32_16x16x4f32(y0[c1].y, y0[c2].y, w, 0, 0, 0);
    u = __builtin_amdgcn_mfma_f32_16x16x4f32(y0[a1].z, y0[a2].z, u, 0, 0, 0);
    w = __builtin_amdgcn_mfma_f32_16x16x4f32(y0[c1].z, y0[c2].z, w, 0, 0, 0);
    u = __builtin_amdgcn_mfma_f32_16x16x4f32(y0[a1].w, y0[a2].w, u, 0, 0, 0);
    w = __builtin_amdgcn_mfma_f32_16x16x4f32(y0[c1].w, y0[c2].w, w, 0, 0, 0);
    u = __builtin_amdgcn_mfma_f32_16x16x4f32(y1[a1].x, y1[a2].x, u, 0, 0, 0);
    w = __builtin_amdgcn_mfma_f32_16x16x4f32(y1[c1].x, y1[c2].x, w, 0, 0, 0);
    u = __builtin_amdgcn_mfma_f32_16x16x4f32(y1[a1].y, y1[a2].y, u, 0, 0, 0);
    w = __builtin_amdgcn_mfma_f32_16x16x4f32(y1[c1].y, y1[c2].y, w, 0, 0, 0);
    u = __builtin_amdgcn_mfma_f32_16x16x4f32(y1[a1].z, y1[a2].z, u, 0, 0, 0);
    w = __builtin_amdgcn_mfma_f32_16x16x4f32(y1[c1].z, y1[c2].z, w, 0, 0, 0);
    u = __builtin_amdgcn_mfma_f32_16x16x4f32(y1[a1].w, y1[a2].w, u, 0, 0, 0);
    w = __builtin_amdgcn_mfma_f32_16x16x4f32(y1[c1].w, y1[c2].w, w, 0, 0, 0);
    gram_flush<NB, q>(u, acc64[I]);
    gram_flush<NB, q2>(w, acc64[I + 1]);
    gram_pairs<NB, PH, I + 2>(y0, y1, acc64);
  } else if constexpr (I < S::PPW && q < S::NBP) {
    constexpr int b1 = pair_b1(NB, q), b2 = pair_b2(NB, q);
    f4 acc = __builtin_amdgcn_mfma_f32_16x16x4f32(y0[b1].x, y0[b2].x, zero, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(y0[b1].y, y0[b2].y, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(y0[b1].z, y0[b2].z, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(y0[b1].w, y0[b2].w, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(y1[b1].x, y1[b2].x, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(y1[b1].y, y1[b2].y, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(y1[b1].z, y1[b2].z, acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(y1[b1].w, y1[b2].w, acc, 0, 0, 0);
    gram_flush<NB, q>(acc, acc64[I]);
  }
}

// This wave's half h of the stage in `buf`, block pairs of parity PH.
template <int NB, int PH>
__device__ __forceinline__ void gram_multiply(const float* __restrict__ buf, int h, int g, int r,
                                              double (*acc64)[4]) {
#pragma unroll
  for (int grp = 0; grp < 8; grp += 2) {
    const int col = 128 * h + 16 * grp + 4 * g;
    f4 y0[NB], y1[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      y0[b] = *reinterpret_cast<const f4*>(buf + (16 * b + r) * kGramPitch + col);
      y1[b] = *reinterpret_cast<const f4*>(buf + (16 * b + r) * kGramPitch + col + 16);
    }
    gram_pairs<NB, PH, 0>(y0, y1, acc64);
  }
}

// The stages of this workgroup: load, stage in LDS, multiply. Workgroups
// 0 .. G-1 take the full stages b, b + G, ...; when kGramStage does not divide
// d, one more workgroup (b = G) takes the partial last stage alone, so that the
// loop over full stages carries no tail handling.
template <int NB, bool PAD, int PH>
__device__ __forceinline__ void gram_tile(const float* __restrict__ x, int n, int64_t d, int ref,
                                          int wave, float* __restrict__ buf, double (*acc64)[4]) {
  using S = GramShape<NB>;
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4, r = lane & 15;
  const int64_t full = d / kGramStage;  // full stages
  const int64_t b = blockIdx.x;
  const int64_t G = gridDim.x - (full * kGramStage < d ? 1 : 0);
  f4 v[S::RPW];
  f4 vr;
  if (b == G) {
    gram_issue<NB, PAD, false>(MatrixRows{x, d}, n, d, ref, wave, lane, full * kGramStage, v, vr);
    lds_barrier();
    gram_put<NB, PAD>(buf, n, wave, lane, v, vr);
    lds_barrier();
    gram_multiply<NB, PH>(buf, wave & 1, g, r, acc64);
    return;
  }
  const int64_t mine = (full > b) ? (full - b + G - 1) / G : 0;
  if (mine > 0)
    gram_issue<NB, PAD, true>(MatrixRows{x, d}, n, d, ref, wave, lane, b * kGramStage, v, vr);
  for (int64_t k = 0; k < mine; ++k) {
    lds_barrier();                    // every wave is done with the previous stage
    gram_put<NB, PAD>(buf, n, wave, lane, v, vr);
    if (k + 1 < mine)                 // in flight during the multiply below
      gram_issue<NB, PAD, true>(MatrixRows{x, d}, n, d, ref, wave, lane,
                                (b + (k + 1) * G) * kGramStage, v, vr);
    lds_barrier();                    // the whole stage is in LDS
    gram_multiply<NB, PH>(buf, wave & 1, g, r, acc64);
  }
}

// Partials of a workgroup: entry q*256 + row*16 + col holds
// G[16*b1 + row][16*b2 + col] (MFMA output: lane l, component e is row
// 4*(l/16) + e, column l%16); the two halves of pair q are held by waves
// 2*(q%2) (h = 0) and 2*(q%2) + 1 and added half 0 first. out[entry * stride].
template <int NB>
__device__ __forceinline__ void gram_write_partials(const double (*acc64)[4], float* buf, int wave,
                                                    int g, int r, double* __restrict__ out,
                                                    int64_t stride) {
  using S = GramShape<NB>;
  __syncthreads();
  double* red = reinterpret_cast<double*>(buf);  // 2 x 256 doubles (4 KB <= buf)
  const int t = threadIdx.x;
#pragma unroll
  for (int q = 0; q < S::NBP; ++q) {
    if ((wave >> 1) == (q & 1)) {
#pragma unroll
      for (int e = 0; e < 4; ++e) red[(wave & 1) * 256 + (4 * g + e) * 16 + r] = acc64[q / 2][e];
    }
    __syncthreads();
    out[(q * 256 + t) * stride] = red[t] + red[256 + t];
    __syncthreads();
  }
}

template <int NB, bool PAD>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(2)))
void k_dist_gram(const float* __restrict__ x, int n, int64_t d,
                 const int32_t* __restrict__ ref_idx, double* __restrict__ partial) {
  using S = GramShape<NB>;
  __shared__ __attribute__((aligned(16))) float buf[S::ROWS * kGramPitch];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4, r = lane & 15;
  const int ref = *ref_idx;
  double acc64[S::PPW][4];
#pragma unroll
  for (int i = 0; i < S::PPW; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e) acc64[i][e] = 0.0;
  if (wave < 2) gram_tile<NB, PAD, 0>(x, n, d, ref, wave, buf, acc64);
  else gram_tile<NB, PAD, 1>(x, n, d, ref, wave, buf, acc64);
  gram_write_partials<NB>(acc64, buf, wave, g, r, partial + blockIdx.x, gridDim.x);
}

// ---------------------------------------------------------------------------
// The Gram engine over a table of segments (segment s of vector i at
// ptrs[s * n + i], dims[s] floats): the stages of all segments of the launch
// form one list (segment s owns stages tab.first[s] .. tab.first[s+1]-1, the
// last one partial when 256 does not divide dims[s]), and workgroup b takes
// stages b, b + G, ... of it, each with its segment's rows. One reference row
// index serves every segment (D is the same whatever row each coordinate is
// shifted by). Tile b of the launch writes column tile_base + b of partials
// with `tiles` columns in all.
template <int NB, bool PAD, int PH>
__device__ __forceinline__ void gram_tile_table(const float* const* __restrict__ ptrs,
                                                const SegTable& tab, int n, int ref, int wave,
                                                float* __restrict__ buf, double (*acc64)[4]) {
  using S = GramShape<NB>;
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4, r = lane & 15;
  const int64_t G = gridDim.x;
  const int64_t total = tab.first[tab.count];
  auto issue = [&](int64_t stage, f4* v, f4& vr) {
    const int sg = seg_of(tab, static_cast<int>(stage));
    const int64_t c0 = (stage - tab.first[sg]) * kGramStage;
    const int64_t d = tab.dims[sg];
    const TableRows src{ptrs + static_cast<int64_t>(sg) * n};
    if (c0 + kGramStage <= d) gram_issue<NB, PAD, true>(src, n, d, ref, wave, lane, c0, v, vr);
    else gram_issue<NB, PAD, false>(src, n, d, ref, wave, lane, c0, v, vr);
  };
  f4 v[S::RPW];
  f4 vr;
  int64_t stage = blockIdx.x;
  if (stage < total) issue(stage, v, vr);
  for (; stage < total; stage += G) {
    lds_barrier();  // every wave is done with the previous stage
    gram_put<NB, PAD>(buf, n, wave, lane, v, vr);
    if (stage + G < total) issue(stage + G, v, vr);  // in flight during the multiply
    lds_barrier();  // the whole stage is in LDS
    gram_multiply<NB, PH>(buf, wave & 1, g, r, acc64);
  }
}

template <int NB, bool PAD>
__global__ __launch_bounds__(kBlock) __attribute__((amdgpu_waves_per_eu(2)))
void k_dist_gram_table(const float* const* __restrict__ ptrs, SegTable tab, int n,
                       const int32_t* __restrict__ ref_idx, int64_t tile_base, int64_t tiles,
                       double* __restrict__ partial) {
  using S = GramShape<NB>;
  __shared__ __attribute__((aligned(16))) float buf[S::ROWS * kGramPitch];
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4, r = lane & 15;
  const int ref = *ref_idx;
  double acc64[S::PPW][4];
#pragma unroll
  for (int i = 0; i < S::PPW; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e) acc64[i][e] = 0.0;
  if (wave < 2) gram_tile_table<NB, PAD, 0>(ptrs, tab, n, ref, wave, buf, acc64);
  else gram_tile_table<NB, PAD, 1>(ptrs, tab, n, ref, wave, buf, acc64);
  gram_write_partials<NB>(acc64, buf, wave, g, r, partial + tile_base + blockIdx.x, tiles);
}

// ---------------------------------------------------------------------------
// Tiles -> entry sums: block e adds partial[e * tiles + t] over all tiles.
// Thread u takes t = u, u + 256, ... in ascending order, then the 256 thread
// sums are combined by a fixed binary tree: the result depends on (tiles)
// only, never on scheduling.
__global__ __launch_bounds__(kBlock) void k_sum_tiles(const double* __restrict__ partial,
                                                      int64_t tiles,
                                                      double* __restrict__ sums) {
  __shared__ double red[kBlock];
  const double* __restrict__ row = partial + static_cast<int64_t>(blockIdx.x) * tiles;
  double a = 0.0;
  int64_t t = threadIdx.x;
  for (; t + 7 * kBlock < tiles; t += 8 * kBlock) {  // eight loads in flight, added in order
    double v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = row[t + u * kBlock];
#pragma unroll
    for (int u = 0; u < 8; ++u) a += v[u];
  }
  for (; t < tiles; t += kBlock) a += row[t];
  red[threadIdx.x] = a;
  __syncthreads();
  for (int h = kBlock / 2; h > 0; h >>= 1) {
    if (threadIdx.x < h) red[threadIdx.x] += red[threadIdx.x + h];
    __syncthreads();
  }
  if (threadIdx.x == 0) sums[blockIdx.x] = red[0];
}

// D (n x n fp64) from the entry sums, for callers that want the matrix.
__global__ __launch_bounds__(kBlock) void k_write_dist(DistSums ds, double* __restrict__ dist) {
  const int n = ds.n;
  for (int idx = threadIdx.x; idx < n * n; idx += kBlock) dist[idx] = dist_entry(ds, idx / n, idx % n);
}

// Segmented aggregation: add one segment's D into the running n x n sum.
__global__ __launch_bounds__(kBlock) void k_accumulate_dist(DistSums ds, double* __restrict__ acc) {
  const int n = ds.n;
  for (int idx = threadIdx.x; idx < n * n; idx += kBlock) acc[idx] += dist_entry(ds, idx / n, idx % n);
}

__global__ __launch_bounds__(kBlock) void k_zero_f64(double* __restrict__ p, int count) {
  for (int idx = threadIdx.x; idx < count; idx += kBlock) p[idx] = 0.0;
}


// ---------------------------------------------------------------------------
template <int N, int W>
hipError_t launch_direct_nw(const float* x, const DistPlan& p, double* partial, double* colsum,
                            hipStream_t s) {
  if constexpr (N <= kColSumMaxN) {
    if (colsum) {
      launch("dist_direct_sum", k_dist_direct_sum<N, W>, dim3(static_cast<unsigned>(p.tiles)),
             dim3(kBlock), 0, s, x, p.d, p.chunk, partial, colsum);
      return hipGetLastError();
    }
  }
  if (colsum) return hipErrorInvalidValue;
  launch("dist_direct", k_dist_direct<N, W>, dim3(static_cast<unsigned>(p.tiles)), dim3(kBlock), 0,
    s, x, p.d, p.chunk, partial);
  return hipGetLastError();
}

// Widest per-lane load that keeps the n(n-1)/2 accumulators and the n x W
// loaded values within the registers of four waves per SIMD (16-byte loads
// stream an n-row read fastest).
int direct_width_cap(int n) { return n <= 12 ? 4 : (n <= 19 ? 2 : 1); }

template <int N>
hipError_t launch_direct_n(const float* x, const DistPlan& p, double* partial, double* colsum,
                           hipStream_t s) {
  if constexpr (N <= 12) {
    if (p.width == 4) return launch_direct_nw<N, 4>(x, p, partial, colsum, s);
  }
  if constexpr (N <= 19) {
    if (p.width >= 2) return launch_direct_nw<N, 2>(x, p, partial, colsum, s);
  }
  return launch_direct_nw<N, 1>(x, p, partial, colsum, s);
}

template <int N>
hipError_t launch_direct_dispatch(int n, const float* x, const DistPlan& p, double* partial,
                                  double* colsum, hipStream_t s) {
  if constexpr (N > kDirectMaxNLimit) {
    return hipErrorInvalidValue;
  } else {
    if (n == N) return launch_direct_n<N>(x, p, partial, colsum, s);
    return launch_direct_dispatch<N + 1>(n, x, p, partial, colsum, s);
  }
}

template <int NB>
hipError_t launch_gram_nb(const float* x, const DistPlan& p, const int32_t* ref, double* partial,
                          hipStream_t s) {
  if (p.n < 16 * NB)
    launch("dist_gram", k_dist_gram<NB, true>, dim3(static_cast<unsigned>(p.tiles)), dim3(kBlock),
           0, s, x, p.n, p.d, ref, partial);
  else
    launch("dist_gram", k_dist_gram<NB, false>, dim3(static_cast<unsigned>(p.tiles)), dim3(kBlock),
           0, s, x, p.n, p.d, ref, partial);
  return hipGetLastError();
}

size_t align256(size_t b) { return (b + 255) & ~static_cast<size_t>(255); }

// Compute units of the current device (256 on MI355X; also the fallback when
// no device is available, e.g. when only planning on a host without a GPU).
int device_cus() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      cus <= 0) {
    (void)hipGetLastError();
    return 256;
  }
  return cus;
}

template <int NB>
int gram_blocks_per_cu_nb() {
  int blocks = 0, blocks_pad = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, k_dist_gram<NB, false>, kBlock, 0) !=
          hipSuccess ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks_pad, k_dist_gram<NB, true>, kBlock,
                                                   0) != hipSuccess ||
      blocks <= 0) {
    (void)hipGetLastError();
    return 2;
  }
  return blocks < blocks_pad ? blocks : blocks_pad;  // the grid fits either variant
}

// Resident workgroups per CU of the Gram kernel for nb row blocks.
int gram_blocks_per_cu(int nb) {
  static int cache[kGramBlocks + 1] = {};
  int& c = cache[nb];
  if (c == 0) {
    switch (nb) {
      case 1: c = gram_blocks_per_cu_nb<1>(); break;
      case 2: c = gram_blocks_per_cu_nb<2>(); break;
      case 3: c = gram_blocks_per_cu_nb<3>(); break;
      default: c = gram_blocks_per_cu_nb<4>(); break;
    }
  }
  return c;
}

// The same for the table kernel.
template <int NB>
int gram_table_blocks_per_cu_nb() {
  int blocks = 0, blocks_pad = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, k_dist_gram_table<NB, false>, kBlock,
                                                   0) != hipSuccess ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks_pad, k_dist_gram_table<NB, true>,
                                                   kBlock, 0) != hipSuccess ||
      blocks <= 0) {
    (void)hipGetLastError();
    return 2;
  }
  return blocks < blocks_pad ? blocks : blocks_pad;
}

int gram_table_blocks_per_cu(int nb) {
  static int cache[kGramBlocks + 1] = {};
  int& c = cache[nb];
  if (c == 0) {
    switch (nb) {
      case 1: c = gram_table_blocks_per_cu_nb<1>(); break;
      case 2: c = gram_table_blocks_per_cu_nb<2>(); break;
      case 3: c = gram_table_blocks_per_cu_nb<3>(); break;
      default: c = gram_table_blocks_per_cu_nb<4>(); break;
    }
  }
  return c;
}

// Launches of the table Gram kernel: at most kSegMax segments each; f(first
// segment, table (first[] in stages), workgroups) for each launch with work.
template <class F>
hipError_t for_each_gram_launch(int n, const int64_t* dims, int K, F&& f) {
  const int nb = (n + 15) / 16;
  const int64_t slots = static_cast<int64_t>(device_cus()) * gram_table_blocks_per_cu(nb);
  for (int g0 = 0; g0 < K; g0 += kSegMax) {
    SegTable tab{};
    tab.count = K - g0 < kSegMax ? K - g0 : kSegMax;
    int64_t total = 0;
    for (int sg = 0; sg < tab.count; ++sg) {
      tab.first[sg] = static_cast<int32_t>(total);
      tab.span[sg] = kGramStage;
      tab.dims[sg] = dims[g0 + sg];
      tab.outs[sg] = nullptr;
      total += (dims[g0 + sg] + kGramStage - 1) / kGramStage;
      if (total > 0x7fffffff) return hipErrorInvalidValue;
    }
    tab.first[tab.count] = static_cast<int32_t>(total);
    if (total == 0) continue;
    const hipError_t e = f(g0, tab, total < slots ? total : slots);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

template <int NB>
hipError_t launch_gram_table_nb(const float* const* ptrs, int n, const SegTable& tab,
                                int64_t groups, const int32_t* ref, int64_t base, int64_t tiles,
                                double* partial, hipStream_t s) {
  if (n < 16 * NB)
    launch("dist_gram_table", k_dist_gram_table<NB, true>, dim3(static_cast<unsigned>(groups)),
           dim3(kBlock), 0, s, ptrs, tab, n, ref, base, tiles, partial);
  else
    launch("dist_gram_table", k_dist_gram_table<NB, false>, dim3(static_cast<unsigned>(groups)),
           dim3(kBlock), 0, s, ptrs, tab, n, ref, base, tiles, partial);
  return hipGetLastError();
}

int g_direct_max_n = 20;

}  // namespace

int64_t table_gram_tiles(const int64_t* dims, int K, int n) {
  int64_t tiles = 0;
  const hipError_t e = for_each_gram_launch(n, dims, K, [&](int, const SegTable&, int64_t groups) {
    tiles += groups;
    return hipSuccess;
  });
  return e == hipSuccess ? tiles : -1;
}

size_t table_gram_probe_bytes() {
  return align256(static_cast<size_t>(kProbeRuns) * kNmax * kNmax * sizeof(double)) +
         align256(sizeof(int32_t));
}

int32_t* table_reference_slot(void* probe_space) {
  return reinterpret_cast<int32_t*>(
      static_cast<char*>(probe_space) +
      align256(static_cast<size_t>(kProbeRuns) * kNmax * kNmax * sizeof(double)));
}

hipError_t enqueue_table_reference(const float* const* ptrs, int n, const int64_t* dims, int K,
                                   void* probe_space, hipStream_t s) {
  // probed on the longest segment (the first of equal ones)
  int big = 0;
  for (int sg = 1; sg < K; ++sg)
    if (dims[sg] > dims[big]) big = sg;
  if (K == 0 || dims[big] == 0) return hipErrorInvalidValue;
  double* probe = static_cast<double*>(probe_space);
  const int runs = probe_runs(dims[big]);
  launch("probe", k_probe<TableRows>, dim3(n, runs), dim3(kBlock), 0, s,
         TableRows{ptrs + static_cast<int64_t>(big) * n}, n, dims[big], probe);
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  launch("pick_ref", k_pick_ref, dim3(1), dim3(kPickThreads), 0, s, probe, n, runs,
         table_reference_slot(probe_space));
  return hipGetLastError();
}

hipError_t enqueue_distances_table_gram(const float* const* ptrs, int n, const int64_t* dims,
                                        int K, double* partial, int64_t tiles, void* probe_space,
                                        hipStream_t s) {
  hipError_t e = enqueue_table_reference(ptrs, n, dims, K, probe_space, s);
  if (e != hipSuccess) return e;
  const int32_t* ref = table_reference_slot(probe_space);
  int64_t base = 0;
  const int nb = (n + 15) / 16;
  return for_each_gram_launch(n, dims, K, [&](int g0, const SegTable& tab, int64_t groups) {
    const float* const* p = ptrs + static_cast<int64_t>(g0) * n;
    hipError_t r;
    switch (nb) {
      case 1: r = launch_gram_table_nb<1>(p, n, tab, groups, ref, base, tiles, partial, s); break;
      case 2: r = launch_gram_table_nb<2>(p, n, tab, groups, ref, base, tiles, partial, s); break;
      case 3: r = launch_gram_table_nb<3>(p, n, tab, groups, ref, base, tiles, partial, s); break;
      case 4: r = launch_gram_table_nb<4>(p, n, tab, groups, ref, base, tiles, partial, s); break;
      default: return hipErrorInvalidValue;
    }
    base += groups;
    return r;
  });
}

int direct_max_n() { return __atomic_load_n(&g_direct_max_n, __ATOMIC_RELAXED); }
void set_direct_max_n(int n) { __atomic_store_n(&g_direct_max_n, n, __ATOMIC_RELAXED); }

int vector_width(const float* p) { return reinterpret_cast<uintptr_t>(p) % 4 == 0 ? 4 : 1; }

// Coordinates per tile of the direct engine: at most kDirectLaneCoords per lane
// (each fp32 accumulator sums at most that many squares before the tile is
// reduced in fp64), fewer when d is small, so that the grid still has about two
// tiles per CU; always a multiple of one pass of the block (kBlock * width).
int64_t direct_chunk(int64_t d, int width) {
  const int64_t pass = static_cast<int64_t>(kBlock) * width;
  const int64_t most = static_cast<int64_t>(kBlock) * kDirectLaneCoords;
  const int64_t want = 2 * static_cast<int64_t>(device_cus());
  int64_t chunk = (d + want - 1) / want;
  chunk = (chunk + pass - 1) / pass * pass;
  return chunk < pass ? pass : (chunk > most ? most : chunk);
}

DistPlan plan_distances(int n, int64_t d, const float* x) {
  DistPlan p;
  p.n = n;
  p.d = d;
  if (n < 2 || d == 0) return p;  // D is all zeros
  if (n <= direct_max_n()) {
    p.engine = kEngineDirect;
    p.width = vector_width(x);
    if (p.width > direct_width_cap(n)) p.width = direct_width_cap(n);
    p.chunk = direct_chunk(d, p.width);
    p.entries = n * (n - 1) / 2;
  } else {
    p.engine = kEngineGram;
    p.width = 4;  // 16-byte loads of 1 KB row runs
    // As many workgroups as the device holds resident (at most one per
    // stage); workgroup b takes stages b, b + tiles, ...
    const int nb = (n + 15) / 16;
    // The partial last stage, if any, takes one workgroup of its own.
    const int64_t slots = static_cast<int64_t>(device_cus()) * gram_blocks_per_cu(nb);
    const int64_t full = d / kGramStage;
    const int64_t tail = full * kGramStage < d ? 1 : 0;
    p.chunk = kGramStage;
    p.entries = nb * (nb + 1) / 2 * 256;
    p.tiles = (full < slots - tail ? full : slots - tail) + tail;
    return p;
  }
  p.tiles = (d + p.chunk - 1) / p.chunk;
  return p;
}

size_t dist_workspace_bytes(const DistPlan& p) {
  size_t b = 0;
  if (p.engine != kEngineNone) {
    b += align256(static_cast<size_t>(p.tiles) * p.entries * sizeof(double));
    b += align256(static_cast<size_t>(p.entries) * sizeof(double));
  }
  if (p.engine == kEngineGram) {
    b += align256(static_cast<size_t>(kProbeRuns) * kNmax * kNmax * sizeof(double));
    b += align256(sizeof(int32_t));
  }
  return b;
}

DistWorkspace carve_dist_workspace(const DistPlan& p, void* base) {
  DistWorkspace w;
  char* c = static_cast<char*>(base);
  if (p.engine != kEngineNone) {
    w.partial = reinterpret_cast<double*>(c);
    c += align256(static_cast<size_t>(p.tiles) * p.entries * sizeof(double));
    w.sums = reinterpret_cast<double*>(c);
    c += align256(static_cast<size_t>(p.entries) * sizeof(double));
  }
  if (p.engine == kEngineGram) {
    w.probe = reinterpret_cast<double*>(c);
    c += align256(static_cast<size_t>(kProbeRuns) * kNmax * kNmax * sizeof(double));
    w.ref = reinterpret_cast<int32_t*>(c);
  }
  return w;
}

DistSums dist_sums(const DistPlan& p, const DistWorkspace& ws) {
  DistSums ds;
  ds.sums = ws.sums;
  ds.engine = p.engine;
  ds.n = p.n;
  return ds;
}

hipError_t enqueue_reference(const float* x, const DistPlan& p, const DistWorkspace& ws,
                             hipStream_t s) {
  const int runs = probe_runs(p.d);
  launch("probe", k_probe<MatrixRows>, dim3(p.n, runs), dim3(kBlock), 0, s, MatrixRows{x, p.d},
         p.n, p.d, ws.probe);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  launch("pick_ref", k_pick_ref, dim3(1), dim3(kPickThreads), 0, s, ws.probe, p.n, runs, ws.ref);
  return hipGetLastError();
}

bool foldable(const DistPlan& p, int max_entries) {
  return p.engine == kEngineDirect && p.tiles <= kFoldTiles && p.entries <= max_entries;
}

hipError_t enqueue_distances(const float* x, const DistPlan& p, const DistWorkspace& ws,
                             hipStream_t s, bool sum_tiles, double* colsum) {
  hipError_t e = hipSuccess;
  if (colsum && (p.engine != kEngineDirect || p.n > kColSumMaxN)) return hipErrorInvalidValue;
  if (p.engine == kEngineNone) return hipSuccess;  // D is all zeros: nothing to compute
  if (p.engine == kEngineDirect) {
    e = launch_direct_dispatch<2>(p.n, x, p, ws.partial, colsum, s);
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
  if (e != hipSuccess || !sum_tiles) return e;
  launch("sum_tiles", k_sum_tiles, dim3(p.entries), dim3(kBlock), 0, s, ws.partial, p.tiles,
    ws.sums);
  return hipGetLastError();
}

hipError_t enqueue_sum_tiles(const double* partial, int64_t tiles, int entries, double* sums,
                             hipStream_t s) {
  launch("sum_tiles", k_sum_tiles, dim3(entries), dim3(kBlock), 0, s, partial, tiles, sums);
  return hipGetLastError();
}

hipError_t enqueue_accumulate_dist(const DistSums& ds, double* acc, hipStream_t s) {
  launch("accumulate_dist", k_accumulate_dist, dim3(1), dim3(kBlock), 0, s, ds, acc);
  return hipGetLastError();
}

hipError_t enqueue_zero_f64(double* p, int count, hipStream_t s) {
  launch("zero", k_zero_f64, dim3(1), dim3(kBlock), 0, s, p, count);
  return hipGetLastError();
}

hipError_t enqueue_write_dist(const DistSums& ds, double* dist, hipStream_t s) {
  launch("write_dist", k_write_dist, dim3(1), dim3(kBlock), 0, s, ds, dist);
  return hipGetLastError();
}

}  // namespace garfield
