// Pairwise squared distances D[i][j] = sum_c (x_ic - x_jc)^2 -- the O(n^2 d)
// step shared by Krum, Multi-Krum, MDA and Bulyan (Section 3.1 items 2-4;
// the paper's complexity discussion in Section 5.3 attributes the quadratic
// growth in n to it).
//
// The coordinates are cut into tiles of `chunk` consecutive coordinates, one
// workgroup per tile. Each tile writes one fp64 partial sum per entry (entry-
// major: partial[entry * tiles + tile]); k_sum_tiles then adds the tiles of
// each entry in a fixed order, so D is deterministic and depends only on
// (n, d), never on scheduling. The consumers build D from the entry sums
// (dist_layout.h). Two engines:
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
#include "dist_layout.h"
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
  block_reduce_pairs<P>(acc, partial + blockIdx.x, gridDim.x);
}

// ---------------------------------------------------------------------------
// Gram engine, step 1: probe. Block i sums (x_i - x_j)^2 for every j over a
// sample of kProbeRuns runs of kBlock consecutive coordinates spread evenly
// over d (all coordinates when d is smaller than the sample), and writes row
// i of the probe matrix (kNmax columns, fp64).
__global__ __launch_bounds__(kBlock) void k_probe(const float* __restrict__ x, int n, int64_t d,
                                                  double* __restrict__ probe) {
  const int i = blockIdx.x;
  float acc[kNmax];
#pragma unroll
  for (int j = 0; j < kNmax; ++j) acc[j] = 0.0f;
  const int64_t sample = static_cast<int64_t>(kProbeRuns) * kBlock;
  const int64_t runs = (d <= sample) ? 1 : kProbeRuns;
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
  block_reduce_pairs<kNmax>(acc, probe + i * kNmax, 1);
}

// Gram engine, step 2: the reference row is the one whose sum of its
// ceil(n/2) smallest probe distances (self included, which is 0) is lowest:
// with an honest majority this is a central, honest row.
__global__ __launch_bounds__(kBlock) void k_pick_ref(const double* __restrict__ probe, int n,
                                                     int32_t* __restrict__ ref) {
  __shared__ double P[kNmax * kNmax];
  __shared__ unsigned char take[kNmax * kNmax];
  __shared__ double score[kNmax];
  for (int idx = threadIdx.x; idx < n * n; idx += kBlock)
    P[idx] = probe[(idx / n) * kNmax + idx % n];
  __syncthreads();
  const int h = (n + 1) / 2;
  // entry (i, j) contributes to row i's score when its rank (ties by index)
  // among row i is below h
  for (int idx = threadIdx.x; idx < n * n; idx += kBlock) {
    const int i = idx / n, j = idx % n;
    const double v = P[idx];
    int rank = 0;
    for (int j2 = 0; j2 < n; ++j2) {
      const double w = P[i * n + j2];
      rank += (w < v) || (w == v && j2 < j);
    }
    take[idx] = rank < h;
  }
  __syncthreads();
  if (threadIdx.x < n) {
    double s = 0.0;
    for (int j = 0; j < n; ++j)
      if (take[threadIdx.x * n + j]) s += P[threadIdx.x * n + j];
    score[threadIdx.x] = s;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    int best = 0;
    for (int j = 1; j < n; ++j)
      if (score[j] < score[best]) best = j;
    *ref = best;
  }
}

// ---------------------------------------------------------------------------
// Gram engine, step 3: G partial sums per tile on MFMA (v_mfma_f32_16x16x4_f32).
//
// The workgroup streams its tile in stages of 64 coordinates. For each stage
// every thread loads 4 consecutive coordinates of up to 4 rows (and of the
// reference row), subtracts the reference, and stores them into one of two
// LDS buffers (row-major, 68-float pitch); while the waves multiply from one
// buffer the next stage's loads are in flight.
//
// The work of a stage is NBP block pairs (b1 <= b2) x 16 k-slices. It is cut
// into UNITS = NBP * H units (pair q, k-part h) with UNITS a multiple of 4,
// and wave w takes units u = w, w + 4, ...: the four waves issue the same
// number of MFMAs. Within a 16-coordinate group lane (g = l / 16, r = l % 16)
// reads row 16b + r, coordinates 4g .. 4g + 3, as one 16-byte LDS read: these
// are the A (or B) operands of 4 consecutive MFMA k-slices. Each fp32
// accumulator takes 4 MFMAs (16 products) before it is added into fp64.
template <int NB>
struct GramShape {
  static constexpr int NBP = NB * (NB + 1) / 2;
  static constexpr int H = (NBP % 4 == 0) ? 1 : ((NBP % 2 == 0) ? 2 : 4);
  static constexpr int UNITS = NBP * H;
  static constexpr int UPW = UNITS / 4;       // units per wave
  static constexpr int GROUPS = 4 / H;        // 16-coordinate groups per unit per stage
};

constexpr int kGramStage = 64;                // coordinates per stage
constexpr int kGramPitch = kGramStage + 4;    // floats per LDS row

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

// Multiply-accumulate this wave's units over one 16-coordinate group.
template <int NB, int WV, int GRP>
__device__ __forceinline__ void gram_group(const float* __restrict__ buf, f4* acc, int g, int r) {
  using S = GramShape<NB>;
#pragma unroll
  for (int i = 0; i < S::UPW; ++i) {
    const int u = WV + 4 * i;
    const int q = u / S::H;
    const int h = u % S::H;
    if (GRP / S::GROUPS != h) continue;  // this group belongs to another k-part
    const int b1 = pair_b1(NB, q), b2 = pair_b2(NB, q);
    const f4 a = *reinterpret_cast<const f4*>(buf + (16 * b1 + r) * kGramPitch + 16 * GRP + 4 * g);
    const f4 b = (b1 == b2) ? a
                            : *reinterpret_cast<const f4*>(buf + (16 * b2 + r) * kGramPitch +
                                                           16 * GRP + 4 * g);
    acc[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.x, b.x, acc[i], 0, 0, 0);
    acc[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.y, b.y, acc[i], 0, 0, 0);
    acc[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.z, b.z, acc[i], 0, 0, 0);
    acc[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(a.w, b.w, acc[i], 0, 0, 0);
  }
}

template <int NB, int WV>
__device__ __forceinline__ void gram_stage(const float* __restrict__ buf, f4* acc,
                                           double (*acc64)[4], int g, int r) {
  using S = GramShape<NB>;
#pragma unroll
  for (int grp = 0; grp < 4; ++grp) {
    switch (grp) {
      case 0: gram_group<NB, WV, 0>(buf, acc, g, r); break;
      case 1: gram_group<NB, WV, 1>(buf, acc, g, r); break;
      case 2: gram_group<NB, WV, 2>(buf, acc, g, r); break;
      default: gram_group<NB, WV, 3>(buf, acc, g, r); break;
    }
    // flush the units that just took this group's 4 MFMAs
#pragma unroll
    for (int i = 0; i < S::UPW; ++i) {
      const int u = WV + 4 * i;
      if (grp / S::GROUPS != u % S::H) continue;
      acc64[i][0] += static_cast<double>(acc[i].x);
      acc64[i][1] += static_cast<double>(acc[i].y);
      acc64[i][2] += static_cast<double>(acc[i].z);
      acc64[i][3] += static_cast<double>(acc[i].w);
      acc[i] = f4{0.0f, 0.0f, 0.0f, 0.0f};
    }
  }
}

// Load (registers) the shifted stage starting at c0: rows lr + 16i, 4
// coordinates at c0 + 4*col. Coordinates at or beyond `end` read as 0.
template <int NB, int W>
__device__ __forceinline__ void gram_load(const float* __restrict__ x, const float* __restrict__ xref,
                                          int n, int64_t d, int64_t c0, int64_t end, int lr,
                                          int col, float (*pv)[4], float* pr) {
  const int64_t c = c0 + 4 * col;
  const bool full = c + 4 <= end;
  if (full) {
#pragma unroll
    for (int u = 0; u < 4; u += W) load_w<W, false>(xref + c + u, pr + u);
  } else {
    load_w_tail<4>(xref + c, end - c, pr);
  }
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    const int row = lr + 16 * i;
    if (row < n) {
      const float* p = x + static_cast<int64_t>(row) * d + c;
      if (full) {
#pragma unroll
        for (int u = 0; u < 4; u += W) load_w<W>(p + u, pv[i] + u);
      } else {
        load_w_tail<4>(p, end - c, pv[i]);
      }
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) pv[i][e] = 0.0f;
    }
  }
}

template <int NB>
__device__ __forceinline__ void gram_store(float* __restrict__ buf, int n, int lr, int col,
                                           float (*pv)[4], const float* pr) {
#pragma unroll
  for (int i = 0; i < NB; ++i) {
    const int row = lr + 16 * i;
    f4 y;
    if (row < n) {
      y = f4{pv[i][0] - pr[0], pv[i][1] - pr[1], pv[i][2] - pr[2], pv[i][3] - pr[3]};
    } else {
      y = f4{0.0f, 0.0f, 0.0f, 0.0f};
    }
    *reinterpret_cast<f4*>(buf + row * kGramPitch + 4 * col) = y;
  }
}

// This workgroup's stages are global stages blockIdx.x, + gridDim.x, ...;
// the last global stage may be partial (zero-filled by gram_load).
template <int NB, int W, int WV>
__device__ __forceinline__ void gram_tile(const float* __restrict__ x, int n, int64_t d,
                                          const float* __restrict__ xref,
                                          float* __restrict__ bufs, double (*acc64)[4]) {
  using S = GramShape<NB>;
  const int t = threadIdx.x;
  const int lane = t & 63;
  const int g = lane >> 4, r = lane & 15;
  const int lr = t >> 4, col = t & 15;  // loading role: row lr + 16i, coordinates 4*col..
  f4 acc[S::UPW];
#pragma unroll
  for (int i = 0; i < S::UPW; ++i) acc[i] = f4{0.0f, 0.0f, 0.0f, 0.0f};
  float pv[NB][4];
  float pr[4];
  const int64_t total = (d + kGramStage - 1) / kGramStage;
  const int64_t b = blockIdx.x, G = gridDim.x;
  const int64_t mine = (total > b) ? (total - b + G - 1) / G : 0;
  if (mine <= 0) return;
  auto stage_end = [d](int64_t c0) { return (c0 + kGramStage < d) ? c0 + kGramStage : d; };
  int64_t c0 = b * kGramStage;
  gram_load<NB, W>(x, xref, n, d, c0, stage_end(c0), lr, col, pv, pr);
  gram_store<NB>(bufs, n, lr, col, pv, pr);
  __syncthreads();
  for (int64_t k = 0; k < mine; ++k) {
    float* cur = bufs + (k & 1) * (64 * kGramPitch);
    float* nxt = bufs + ((k + 1) & 1) * (64 * kGramPitch);
    const bool more = k + 1 < mine;
    if (more) {
      c0 = (b + (k + 1) * G) * kGramStage;
      gram_load<NB, W>(x, xref, n, d, c0, stage_end(c0), lr, col, pv, pr);
    }
    gram_stage<NB, WV>(cur, acc, acc64, g, r);
    if (more) gram_store<NB>(nxt, n, lr, col, pv, pr);
    __syncthreads();
  }
}

template <int NB, int W>
__global__ __launch_bounds__(kBlock) void k_dist_gram2(const float* __restrict__ x, int n,
                                                        int64_t d, int64_t chunk,
                                                        const int32_t* __restrict__ ref_idx,
                                                        double* __restrict__ partial) {
  using S = GramShape<NB>;
  __shared__ __attribute__((aligned(16))) float bufs[2 * 64 * kGramPitch];
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4, r = lane & 15;
  const float* __restrict__ xref = x + static_cast<int64_t>(*ref_idx) * d;
  (void)chunk;
  double acc64[S::UPW][4];
#pragma unroll
  for (int i = 0; i < S::UPW; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e) acc64[i][e] = 0.0;
  switch (wave) {
    case 0: gram_tile<NB, W, 0>(x, n, d, xref, bufs, acc64); break;
    case 1: gram_tile<NB, W, 1>(x, n, d, xref, bufs, acc64); break;
    case 2: gram_tile<NB, W, 2>(x, n, d, xref, bufs, acc64); break;
    default: gram_tile<NB, W, 3>(x, n, d, xref, bufs, acc64); break;
  }
  // Combine the k-parts of each pair in ascending h (fixed order) and write the
  // tile's partials: entry q*256 + row*16 + col holds G[16*b1 + row][16*b2 + col].
  double* red = reinterpret_cast<double*>(bufs);  // H x 256 doubles
  double* __restrict__ out = partial + blockIdx.x;
  const int64_t stride = gridDim.x;
#pragma unroll
  for (int q = 0; q < S::NBP; ++q) {
#pragma unroll
    for (int h = 0; h < S::H; ++h) {
      const int u = q * S::H + h;
      if (wave == u % 4) {
#pragma unroll
        for (int e = 0; e < 4; ++e) red[h * 256 + (4 * g + e) * 16 + r] = acc64[u / 4][e];
      }
    }
    __syncthreads();
    const int t = threadIdx.x;
    double v = red[t];
#pragma unroll
    for (int h = 1; h < S::H; ++h) v += red[h * 256 + t];
    out[(q * 256 + t) * stride] = v;
    __syncthreads();
  }
}

// ---------------------------------------------------------------------------
// Gram engine, step 3 for 16-byte-aligned rows: the same contraction with the
// stages brought into LDS by direct global-to-LDS loads (global_load_lds_dwordx4),
// through a ring of three stage buffers, so two stages are in flight while the
// waves multiply the third, with no staging registers.
//
// A stage is 16*NB rows x 16 chunks of 4 coordinates. Chunk c of row `row`
// sits in LDS slot row*17 + c (16 bytes per slot; slot 16 of each row is
// padding), so the 16 rows a fragment read touches fall in distinct bank
// groups, and every fragment address is one per-lane base plus a constant. A
// direct load writes 64 consecutive slots per instruction (lane l -> slot
// base + l); lanes whose slot is padding, or whose row is at or beyond n, load
// row 0 instead (always in bounds) and those rows are masked at use, so every
// lane issues every load and each wave's count of loads in flight is a
// compile-time constant. The shift by the reference row (one of the staged
// rows) is applied when a fragment is read. A final stage that runs past the
// tile end is staged through registers with zero fill.
typedef __attribute__((address_space(3))) void* lds_ptr;

// global_load_lds_dwordx4: 16 bytes per lane from `src` into LDS at
// lds_base + 16 * lane. Written as inline assembly so that the compiler does
// not add a wait for these loads before every later LDS read (it cannot tell
// the ring buffers apart); the ring code waits for them explicitly.
__device__ __forceinline__ void load_lds_16(const float* src, float* lds_base) {
  const lds_ptr lds = (lds_ptr)lds_base;
  const uint32_t m0 = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>((uintptr_t)lds));
  asm volatile(
      "s_mov_b32 m0, %0\n\t"
      "s_nop 0\n\t"
      "global_load_lds_dwordx4 %1, off"
      :
      : "s"(m0), "v"(src)
      : "memory", "m0");
}

template <int NB>
struct Ring {
  static constexpr int SLOTS = 16 * NB * 17;            // 16-byte slots per stage
  static constexpr int LOADS = (SLOTS + 63) / 64;       // load instructions per stage
  static constexpr int FLOATS = LOADS * 64 * 4;         // floats per ring buffer
  // loads per stage issued by wave w (instructions j = w, w + 4, ...)
  __host__ __device__ static constexpr int loads_of(int w) { return (LOADS - w + 3) / 4; }
};

__device__ __forceinline__ int ring_slot(int row, int chunk) { return row * 17 + chunk; }

// Wait until at most N vector-memory operations of this wave are outstanding
// and all of its LDS operations are done (s_waitcnt vmcnt(N) lgkmcnt(0)).
template <int N>
__device__ __forceinline__ void wait_vmem_lds() {
  static_assert(N >= 0 && N < 16, "vmcnt immediate");
  __builtin_amdgcn_s_waitcnt(N | (0x7 << 4) | (0x0 << 8));
}

// Issue the loads of the full stage starting at c0 into `slot` (one buffer).
template <int NB, int WV>
__device__ __forceinline__ void ring_issue(const float* __restrict__ x, int n, int64_t d,
                                           int64_t c0, float* slot) {
  const int l = threadIdx.x & 63;
#pragma unroll
  for (int j = WV; j < Ring<NB>::LOADS; j += 4) {
    const int s = 64 * j + l;
    const int row = s / 17, chunk = s % 17;
    const bool real = chunk < 16 && row < n && row < 16 * NB;
    const float* src = real ? x + static_cast<int64_t>(row) * d + c0 + 4 * chunk : x + c0;
    load_lds_16(src, slot + j * 256);
  }
}

// The last, partial stage [c0, t1) through registers, zero-filled beyond t1
// and for rows at or beyond n.
template <int NB>
__device__ __noinline__ void ring_fill_tail(const float* __restrict__ x, int n, int64_t d,
                                            int64_t c0, int64_t t1, float* slot) {
  for (int s = threadIdx.x; s < Ring<NB>::SLOTS; s += kBlock) {
    const int row = s / 17, chunk = s % 17;
    f4 v = f4{0.0f, 0.0f, 0.0f, 0.0f};
    if (chunk < 16 && row < n) {
      const int64_t c = c0 + 4 * chunk;
      const float* src = x + static_cast<int64_t>(row) * d + c;
      v.x = (c + 0 < t1) ? src[0] : 0.0f;
      v.y = (c + 1 < t1) ? src[1] : 0.0f;
      v.z = (c + 2 < t1) ? src[2] : 0.0f;
      v.w = (c + 3 < t1) ? src[3] : 0.0f;
    }
    *reinterpret_cast<f4*>(slot + 4 * s) = v;
  }
}

// Blocks (16-row groups) that wave WV's units touch in 16-coordinate group GRP.
template <int NB, int WV, int GRP>
__host__ __device__ constexpr unsigned ring_blocks_used() {
  using S = GramShape<NB>;
  unsigned mask = 0;
  for (int i = 0; i < S::UPW; ++i) {
    const int u = WV + 4 * i;
    if (GRP / S::GROUPS != u % S::H) continue;
    mask |= 1u << pair_b1(NB, u / S::H);
    mask |= 1u << pair_b2(NB, u / S::H);
  }
  return mask;
}

// Multiply-accumulate this wave's units over 16-coordinate group GRP: each
// block's shifted fragment is read once and shared by the units using it; the
// first of a unit's 4 MFMAs starts from zero, and the 4 are then added into
// fp64 (16 products per fp32 accumulation).
template <int NB, int WV, int GRP>
__device__ __forceinline__ void ring_group(const float* __restrict__ slot, int n, int ref,
                                           double (*acc64)[4], int g, int r) {
  using S = GramShape<NB>;
  constexpr unsigned used = ring_blocks_used<NB, WV, GRP>();
  if constexpr (used != 0) {
    const int c = 4 * GRP + g;
    const f4 rf = *reinterpret_cast<const f4*>(slot + 4 * ring_slot(ref, c));
    f4 fr[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      if (!((used >> b) & 1u)) continue;
      const int row = 16 * b + r;
      fr[b] = *reinterpret_cast<const f4*>(slot + 4 * ring_slot(row, c)) - rf;
      if (row >= n) fr[b] = f4{0.0f, 0.0f, 0.0f, 0.0f};
    }
    const f4 zero = f4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int i = 0; i < S::UPW; ++i) {
      const int u = WV + 4 * i;
      if (GRP / S::GROUPS != u % S::H) continue;
      const int b1 = pair_b1(NB, u / S::H), b2 = pair_b2(NB, u / S::H);
      f4 acc = __builtin_amdgcn_mfma_f32_16x16x4f32(fr[b1].x, fr[b2].x, zero, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(fr[b1].y, fr[b2].y, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(fr[b1].z, fr[b2].z, acc, 0, 0, 0);
      acc = __builtin_amdgcn_mfma_f32_16x16x4f32(fr[b1].w, fr[b2].w, acc, 0, 0, 0);
      acc64[i][0] += static_cast<double>(acc.x);
      acc64[i][1] += static_cast<double>(acc.y);
      acc64[i][2] += static_cast<double>(acc.z);
      acc64[i][3] += static_cast<double>(acc.w);
    }
  }
}

template <int NB, int WV>
__device__ __forceinline__ void ring_compute(const float* __restrict__ slot, int n, int ref,
                                             double (*acc64)[4], int g, int r) {
  // sched_barrier: keep each group's LDS reads next to their MFMAs
  ring_group<NB, WV, 0>(slot, n, ref, acc64, g, r);
  __builtin_amdgcn_sched_barrier(0);
  ring_group<NB, WV, 1>(slot, n, ref, acc64, g, r);
  __builtin_amdgcn_sched_barrier(0);
  ring_group<NB, WV, 2>(slot, n, ref, acc64, g, r);
  __builtin_amdgcn_sched_barrier(0);
  ring_group<NB, WV, 3>(slot, n, ref, acc64, g, r);
}

// One ring step: wait for stage st (held by `cur`), then refill the buffer
// freed by stage st - 1 (`next`) with stage st + 2, then multiply stage st.
// The barrier is a bare s_barrier: each wave first waits for its own loads of
// stage st (its loads of stage st + 1 may stay in flight) and its LDS
// operations, so after the barrier every wave's part of stage st is in LDS,
// and every wave has finished reading stage st - 1. (A full __syncthreads()
// would also drain the loads of stage st + 1.)
template <int NB, int WV>
__device__ __forceinline__ void ring_step(const float* __restrict__ x, int n, int64_t d,
                                          int64_t k, int64_t mine, int64_t b, int64_t G,
                                          const float* cur, float* next, int ref,
                                          double (*acc64)[4], int g, int r) {
  if (k >= mine) return;
  if (k + 1 < mine) wait_vmem_lds<Ring<NB>::loads_of(WV)>(); else wait_vmem_lds<0>();
  __builtin_amdgcn_s_barrier();
  if (k + 2 < mine) ring_issue<NB, WV>(x, n, d, (b + (k + 2) * G) * kGramStage, next);
  ring_compute<NB, WV>(cur, n, ref, acc64, g, r);
}

// This workgroup's stages: global stages blockIdx.x, + gridDim.x, ... (all
// workgroups stream one compact window of every row at a time, which keeps
// the pages in flight few). The final partial stage (when 64 does not divide
// d) belongs to workgroup (d / 64) % gridDim.x and is taken after the ring.
template <int NB, int WV>
__device__ __forceinline__ void ring_tile(const float* __restrict__ x, int n, int64_t d, int ref,
                                          float* s0, float* s1, float* s2, double (*acc64)[4]) {
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4, r = lane & 15;
  const int64_t full = d / kGramStage;
  const int64_t b = blockIdx.x, G = gridDim.x;
  const int64_t mine = (full > b) ? (full - b + G - 1) / G : 0;  // full stages of this group
  if (mine > 0) ring_issue<NB, WV>(x, n, d, (b + 0 * G) * kGramStage, s0);
  if (mine > 1) ring_issue<NB, WV>(x, n, d, (b + 1 * G) * kGramStage, s1);
  for (int64_t k = 0; k < mine; k += 3) {
    ring_step<NB, WV>(x, n, d, k, mine, b, G, s0, s2, ref, acc64, g, r);
    ring_step<NB, WV>(x, n, d, k + 1, mine, b, G, s1, s0, ref, acc64, g, r);
    ring_step<NB, WV>(x, n, d, k + 2, mine, b, G, s2, s1, ref, acc64, g, r);
  }
  if (full * kGramStage < d && full % G == b) {
    __syncthreads();  // every wave is done with the ring buffers
    ring_fill_tail<NB>(x, n, d, full * kGramStage, d, s0);
    __syncthreads();
    ring_compute<NB, WV>(s0, n, ref, acc64, g, r);
  }
}

template <int NB>
__global__ __launch_bounds__(kBlock) void k_dist_gram_lds(const float* __restrict__ x, int n,
                                                           int64_t d, int64_t chunk,
                                                           const int32_t* __restrict__ ref_idx,
                                                           double* __restrict__ partial) {
  using S = GramShape<NB>;
  __shared__ __attribute__((aligned(16))) float s0[Ring<NB>::FLOATS];
  __shared__ __attribute__((aligned(16))) float s1[Ring<NB>::FLOATS];
  __shared__ __attribute__((aligned(16))) float s2[Ring<NB>::FLOATS];
  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4, r = lane & 15;
  const int ref = *ref_idx;
  (void)chunk;
  double acc64[S::UPW][4];
#pragma unroll
  for (int i = 0; i < S::UPW; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e) acc64[i][e] = 0.0;
  switch (wave) {
    case 0: ring_tile<NB, 0>(x, n, d, ref, s0, s1, s2, acc64); break;
    case 1: ring_tile<NB, 1>(x, n, d, ref, s0, s1, s2, acc64); break;
    case 2: ring_tile<NB, 2>(x, n, d, ref, s0, s1, s2, acc64); break;
    default: ring_tile<NB, 3>(x, n, d, ref, s0, s1, s2, acc64); break;
  }
  __syncthreads();
  // Combine the k-parts of each pair in ascending h (fixed order), one part at
  // a time through a 256-double window of s0, and write the tile's partials:
  // entry q*256 + row*16 + col holds G[16*b1 + row][16*b2 + col].
  double* red = reinterpret_cast<double*>(s0);  // 256 doubles (2 KB <= every ring buffer)
  double* __restrict__ out = partial + blockIdx.x;
  const int64_t stride = gridDim.x;
  const int t = threadIdx.x;
#pragma unroll
  for (int q = 0; q < S::NBP; ++q) {
    double v = 0.0;
#pragma unroll
    for (int h = 0; h < S::H; ++h) {
      const int u = q * S::H + h;
      if (wave == u % 4) {
#pragma unroll
        for (int e = 0; e < 4; ++e) red[(4 * g + e) * 16 + r] = acc64[u / 4][e];
      }
      __syncthreads();
      v += red[t];
      __syncthreads();
    }
    out[(q * 256 + t) * stride] = v;
  }
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
  for (int64_t t = threadIdx.x; t < tiles; t += kBlock) a += row[t];
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


// ---------------------------------------------------------------------------
template <int N, int W>
hipError_t launch_direct_nw(const float* x, const DistPlan& p, double* partial, hipStream_t s) {
  launch("dist_direct", k_dist_direct<N, W>, dim3(static_cast<unsigned>(p.tiles)), dim3(kBlock), 0,
    s, x, p.d, p.chunk, partial);
  return hipGetLastError();
}

// Widest per-lane load that keeps the n(n-1)/2 accumulators and the n x W
// loaded values within the registers of four waves per SIMD (16-byte loads
// stream an n-row read fastest).
int direct_width_cap(int n) { return n <= 12 ? 4 : (n <= 16 ? 2 : 1); }

template <int N>
hipError_t launch_direct_n(const float* x, const DistPlan& p, double* partial, hipStream_t s) {
  if constexpr (N <= 12) {
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
  if constexpr (W == 4) {
    launch("dist_gram", k_dist_gram_lds<NB>, dim3(static_cast<unsigned>(p.tiles)), dim3(kBlock), 0,
           s, x, p.n, p.d, p.chunk, ref, partial);
  } else {
    launch("dist_gram", k_dist_gram2<NB, W>, dim3(static_cast<unsigned>(p.tiles)), dim3(kBlock), 0,
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

template <int NB, int W>
int gram_blocks_per_cu_nw() {
  int blocks = 0;
  hipError_t e;
  if constexpr (W == 4) {
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, k_dist_gram_lds<NB>, kBlock, 0);
  } else {
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, k_dist_gram2<NB, W>, kBlock, 0);
  }
  if (e != hipSuccess || blocks <= 0) {
    (void)hipGetLastError();
    return 2;
  }
  return blocks;
}

// Resident workgroups per CU of the Gram kernel for (nb, width).
int gram_blocks_per_cu(int nb, int width) {
  static int cache[5][5] = {};
  int& c = cache[nb][width];
  if (c == 0) {
    int v = 2;
    switch (nb * 8 + width) {
      case 1 * 8 + 1: v = gram_blocks_per_cu_nw<1, 1>(); break;
      case 1 * 8 + 2: v = gram_blocks_per_cu_nw<1, 2>(); break;
      case 1 * 8 + 4: v = gram_blocks_per_cu_nw<1, 4>(); break;
      case 2 * 8 + 1: v = gram_blocks_per_cu_nw<2, 1>(); break;
      case 2 * 8 + 2: v = gram_blocks_per_cu_nw<2, 2>(); break;
      case 2 * 8 + 4: v = gram_blocks_per_cu_nw<2, 4>(); break;
      case 3 * 8 + 1: v = gram_blocks_per_cu_nw<3, 1>(); break;
      case 3 * 8 + 2: v = gram_blocks_per_cu_nw<3, 2>(); break;
      case 3 * 8 + 4: v = gram_blocks_per_cu_nw<3, 4>(); break;
      case 4 * 8 + 1: v = gram_blocks_per_cu_nw<4, 1>(); break;
      case 4 * 8 + 2: v = gram_blocks_per_cu_nw<4, 2>(); break;
      case 4 * 8 + 4: v = gram_blocks_per_cu_nw<4, 4>(); break;
      default: break;
    }
    c = v;
  }
  return c;
}

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

int vector_width(const float* p) { return reinterpret_cast<uintptr_t>(p) % 4 == 0 ? 4 : 1; }

DistPlan plan_distances(int n, int64_t d, const float* x) {
  DistPlan p;
  p.n = n;
  p.d = d;
  if (n < 2 || d == 0) return p;  // D is all zeros
  if (n <= direct_max_n()) {
    p.engine = kEngineDirect;
    p.width = vector_width(x);
    if (p.width > direct_width_cap(n)) p.width = direct_width_cap(n);
    // kDirectLaneCoords coordinates per lane per tile: each fp32 accumulator
    // sums at most that many squares before the tile is reduced in fp64.
    p.chunk = static_cast<int64_t>(kBlock) * kDirectLaneCoords;
    p.entries = n * (n - 1) / 2;
  } else {
    p.engine = kEngineGram;
    p.width = load_width(x, d);
    // As many workgroups as the device holds resident (at most one per
    // 64-coordinate stage); workgroup b takes stages b, b + tiles, ...
    const int nb = (n + 15) / 16;
    const int64_t slots = static_cast<int64_t>(device_cus()) * gram_blocks_per_cu(nb, p.width);
    const int64_t stages = (d + kGramStage - 1) / kGramStage;
    p.chunk = kGramStage;
    p.entries = nb * (nb + 1) / 2 * 256;
    p.tiles = stages < slots ? stages : slots;
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
    b += align256(static_cast<size_t>(kNmax) * kNmax * sizeof(double));
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
    c += align256(static_cast<size_t>(kNmax) * kNmax * sizeof(double));
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
  launch("probe", k_probe, dim3(p.n), dim3(kBlock), 0, s, x, p.n, p.d, ws.probe);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  launch("pick_ref", k_pick_ref, dim3(1), dim3(kBlock), 0, s, ws.probe, p.n, ws.ref);
  return hipGetLastError();
}

hipError_t enqueue_distances(const float* x, const DistPlan& p, const DistWorkspace& ws,
                             hipStream_t s) {
  hipError_t e = hipSuccess;
  if (p.engine == kEngineNone) return hipSuccess;  // D is all zeros: nothing to compute
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
  launch("sum_tiles", k_sum_tiles, dim3(p.entries), dim3(kBlock), 0, s, ws.partial, p.tiles,
    ws.sums);
  return hipGetLastError();
}

hipError_t enqueue_write_dist(const DistSums& ds, double* dist, hipStream_t s) {
  launch("write_dist", k_write_dist, dim3(1), dim3(kBlock), 0, s, ds, dist);
  return hipGetLastError();
}

}  // namespace garfield
