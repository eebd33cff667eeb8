// Pairwise squared distances D[i][j] = sum_c (x_ic - x_jc)^2 -- the O(n^2 d)
// step shared by Krum, Multi-Krum, MDA and Bulyan (Section 3.1 items 2-4;
// the paper's complexity discussion in Section 6.3 attributes the quadratic
// growth in n to it).
//
// Every workgroup of the distance kernel is a tile: the direct engine cuts the
// coordinates into tiles of `chunk` consecutive coordinates, the Gram engine
// gives each workgroup the 256-coordinate stages s, s + G, s + 2G, ... of its
// slot s (gram_slot: a permutation of the workgroups by XCD). Each tile
// writes one fp64 partial sum per entry (entry-major: partial[entry * tiles +
// tile]); k_sum_tiles then adds the tiles of each entry in a fixed order, so D
// is deterministic and depends only on (n, d), never on scheduling. The
// consumers build D from the entry sums (dist_layout.h). Two engines:
//
//  * direct (n <= direct_max_n(), default 20): every lane accumulates (x_i - x_j)^2 for all
//    n(n-1)/2 pairs in fp32 registers over its coordinates. No cancellation,
//    and identical rows give bit-identical rows of D.
//  * Gram (larger n): G = Y Y^T with Y = X - x_ref (a per-coordinate shift by
//    one input row, chosen robustly by a small probe), each row of Y rounded
//    per 256-coordinate stage to 22-bit integers and multiplied exactly on
//    integer MFMA (v_mfma_i32_16x16x64_i8 on three int8 digits, 16-row
//    blocks, upper block triangle only), then D_ij = G_ii + G_jj - 2 G_ij in
//    fp64. Shifting by a central row keeps the rounding steps, and the
//    cancellation in that difference, small. The products are exact, so
//    identical rows give identical G and D rows and an exact 0 between them,
//    whatever blocks they sit in.

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
// Gram engine, step 3: partial sums of G = Y Y^T, Y = X - x_ref, computed
// exactly on integer MFMA (v_mfma_i32_16x16x64_i8), upper block triangle only.
//
// Streaming and roles. A stage is the 16*NB rows (rows at or beyond n are
// not loaded; their Y rows are 0) times kGramStage = 256 consecutive
// coordinates: 1 KB of every row, the shortest run that streams well from
// rows whose starts are not cache-line aligned (row i starts at i * d
// floats). A workgroup is twelve waves in two roles. Waves 0-7 produce:
// wave w loads rows w*2NB .. w*2NB + 2NB - 1 with one 16-byte load per lane
// per row (lane l: coordinates 4l .. 4l+3, so one instruction reads 1 KB of
// one row), quantizes them into one of two LDS stage buffers, and keeps the
// next DEPTH stages' loads in flight in DEPTH register sets (each row's next
// load is issued as soon as the row is written). Waves 8-11 consume: they
// multiply the stage in the other buffer. One barrier per stage hands the
// buffers over, so quantizing (VALU) and multiplying (matrix cores) overlap
// on every SIMD, which holds two producer waves and one consumer.
//
// Quantizing. y = fl(x - x_ref) in fp32 (one rounding). Per row and stage,
// with E the exponent of the largest |y| (-126 for a zero or subnormal
// maximum) and k = min(21 - E, 127), every y becomes the integer
// q = RNE(y * 2^k), |q| <= 2^22: an error of at most 2^-k / 2, i.e. about
// 2^-23 of the row's largest value in the stage. q is written as three signed
// base-256 digits, q = 65536 a + 256 b + c with c, b in [-128, 127] and a in
// [-64, 64], one int8 plane per digit in LDS (c is q's low byte, b the second
// byte of q + 128, a the third byte of q + 32896), with k per row.
//
// Multiplying. The nine digit products of a block pair go into five int32
// accumulators by weight (aa': 2^32; ab' + ba': 2^24; ac' + bb' + ca': 2^16;
// bc' + cb': 2^8; cc': 1), each product of int8 digits exact and every sum
// exact in int32 (at most 2^23 over a stage). Per stage the five are combined
// in fp64 (a Horner sum in 256, exact: the total is below 2^52) and scaled by
// 2^-(k_i + k_j) (exact), so the stage's G_ij is the exact dot product of the
// two quantized rows; it is then added into an fp64 accumulator. Exactness
// makes the order of the products irrelevant: identical rows give identical
// G rows wherever they sit in the blocks, and an exact 0 between them.
// Consumer wave c takes the block pairs q = c, c + 4, ... over the whole
// stage (K chunks of 64 coordinates: lane (g = l/16, r = l%16) supplies
// coordinates 16g .. 16g+15 of the chunk for row r of the block, in A and in
// B alike).
//
// Partials. Each consumer wave writes the fp64 sums of its pairs as this
// workgroup's partials; the workgroup of slot s takes stages s, s + G, ...
// (G = grid size, one workgroup per CU), so at any time the grid streams one
// compact window of every row.
constexpr int kGramStage = 256;                  // coordinates per stage
// Bytes per LDS row of a digit plane: with 288 the 16-byte fragment reads of
// the multiply (16 rows x 4 column groups per instruction) hit no bank twice
// on gfx950 (measured: 272, 304, 336 and 400 do).
constexpr int kPlanePitch = kGramStage + 32;
// Producer waves (then 4 consumer waves): eight, so that each holds few rows
// and three stages of loads fit beside the consumers' registers at three
// waves per SIMD (four producers with two stages in flight streamed slower).
constexpr int kGramProducers = 8;
constexpr int kGramThreads = (kGramProducers + 4) * 64;
constexpr int kGramWavesPerSimd = (kGramProducers + 4) / 4;
constexpr float kRoundMagic = 12582912.0f;       // 1.5 * 2^23

typedef int i4 __attribute__((ext_vector_type(4)));

template <int NB>
struct GramShape {
  static constexpr int ROWS = 16 * NB;
  static constexpr int NBP = NB * (NB + 1) / 2;   // block pairs b1 <= b2
  static constexpr int RPW = ROWS / kGramProducers;  // rows loaded per producer wave
  static constexpr int PPW = (NBP + 3) / 4;       // pairs per wave (q = w, w + 4, ...)
  static constexpr int PLANE = ROWS * kPlanePitch;  // bytes per digit plane
  static constexpr int BUF = 3 * PLANE + 4 * ROWS;  // three planes, then k per row
  static constexpr int LDS = 2 * BUF;               // two stage buffers
  // stages a producer keeps in flight (register sets of RPW + 1 loads): at
  // n = 64 three stages of 64 KB per CU stream 7% faster than two, and four
  // exceed the registers of three waves per SIMD
  static constexpr int DEPTH = 3;
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

// One 16-byte load of row `row` at coordinate c (lane l of the wave reads
// c = c0 + 4l .. c0 + 4l + 3), coordinates at or beyond d reading as 0 unless
// the stage is known to be whole.
template <bool FULL, class Src>
__device__ __forceinline__ f4 gram_load(const Src& src, int row, int64_t c, int64_t d) {
  const float* p = src.row(row) + c;
  float t[4];
  if constexpr (FULL) {
    load_w<4>(p, t);
  } else {
    if (c + 4 <= d) load_w<4>(p, t); else load_w_tail<4>(p, d - c, t);
  }
  return f4{t[0], t[1], t[2], t[3]};
}

// One stage: its rows, its first coordinate and the length of its segment;
// `full` when all 256 coordinates lie in the segment (wave-uniform).
template <class Src>
struct StageRef {
  Src src;
  int64_t c0;
  int64_t d;
  bool full;
};

// Load row `row` of stage st into out (this lane's 4 coordinates), guarded
// when the stage is partial.
template <class Src>
__device__ __forceinline__ void stage_load(const StageRef<Src>& st, int row, int lane, f4& out) {
  const int64_t c = st.c0 + 4 * lane;
  if (st.full) out = gram_load<true>(st.src, row, c, st.d);
  else out = gram_load<false>(st.src, row, c, st.d);
}

// The row a producer lane loads for row `row` of a whole stage: a padding
// row (at or beyond n) loads the reference row again (an L2 hit; its values
// are replaced by 0), so that every load is issued unconditionally and the
// compiler can count the loads in flight.
template <bool PAD>
__device__ __forceinline__ int load_row(int row, int n, int ref) {
  return (PAD && row >= n) ? ref : row;
}

// Issue the loads of stage st: producer wave pw's rows into v, the reference
// row into vr. WHOLE: st is a full stage, every load unconditional.
template <int NB, bool PAD, bool WHOLE, class Src>
__device__ __forceinline__ void gram_issue(const StageRef<Src>& st, int n, int ref, int pw,
                                           int lane, f4* v, f4& vr) {
  using S = GramShape<NB>;
  const int64_t c = st.c0 + 4 * lane;
#pragma unroll
  for (int i = 0; i < S::RPW; ++i) {
    const int row = pw * S::RPW + i;  // wave-uniform
    if constexpr (WHOLE) v[i] = gram_load<true>(st.src, load_row<PAD>(row, n, ref), c, st.d);
    else if (!PAD || row < n) stage_load(st, row, lane, v[i]);
  }
  if constexpr (WHOLE) vr = gram_load<true>(st.src, ref, c, st.d);
  else stage_load(st, ref, lane, vr);
}

// Per-row maxima of P values per lane (P a power of two, at most 16) over the
// whole wave, transposed: each step pairs a lane with one whose lane bit s
// differs (xor 1, xor 2 by quad permutes, then rotations by 4 and 8 within a
// row of 16 lanes, which also pair opposite bits), and every lane keeps the
// half of its values that its bit s selects, so the count halves per step.
// Then the four rows of 16 lanes are combined by the cross-row swaps. Lane l
// ends with the maximum of value rho(l) over all 64 lanes, where rho(l) is
// the bit reversal of l mod P over log2(P) bits.
template <int CTRL>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t x) {
  return static_cast<uint32_t>(
      __builtin_amdgcn_update_dpp(0, static_cast<int>(x), CTRL, 0xF, 0xF, false));
}

template <int CTRL, int H>
__device__ __forceinline__ void transpose_step(uint32_t* m, bool hi) {
#pragma unroll
  for (int j = 0; j < H; ++j) {
    const uint32_t keep = hi ? m[j + H] : m[j];
    const uint32_t send = hi ? m[j] : m[j + H];
    const uint32_t got = dpp_u32<CTRL>(send);
    m[j] = keep > got ? keep : got;
  }
}

__device__ __forceinline__ uint32_t max_u32(uint32_t a, uint32_t b) { return a > b ? a : b; }

template <int P>
__device__ __forceinline__ uint32_t transpose_max(uint32_t* m, int lane) {
  static_assert(P == 4 || P == 8 || P == 16, "4, 8 or 16 values per lane");
  transpose_step<0xB1, P / 2>(m, lane & 1);           // quad_perm [1, 0, 3, 2]
  transpose_step<0x4E, P / 4>(m, (lane >> 1) & 1);    // quad_perm [2, 3, 0, 1]
  uint32_t u;
  if constexpr (P >= 8) {
    transpose_step<0x124, P / 8>(m, (lane >> 2) & 1); // row_ror 4
    if constexpr (P == 16) {
      transpose_step<0x128, 1>(m, (lane >> 3) & 1);   // row_ror 8
      u = m[0];
    } else {
      u = m[0];
      u = max_u32(u, dpp_u32<0x128>(u));
    }
  } else {
    u = m[0];
    u = max_u32(u, dpp_u32<0x124>(u));
    u = max_u32(u, dpp_u32<0x128>(u));
  }
  const auto s16 = __builtin_amdgcn_permlane16_swap(u, u, false, false);  // rows 0 <-> 1, 2 <-> 3
  u = max_u32(s16[0], s16[1]);
  const auto s32 = __builtin_amdgcn_permlane32_swap(u, u, false, false);  // halves
  return max_u32(s32[0], s32[1]);
}

__host__ __device__ constexpr int bit_reverse(int x, int bits) {
  int r = 0;
  for (int b = 0; b < bits; ++b) r |= ((x >> b) & 1) << (bits - 1 - b);
  return r;
}

typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));

// The two low digit planes of four words: bytes 0 of w (c) and bytes 1 of
// w + 128 (b). The low halves of two words are paired first, so that one
// packed 16-bit add takes the + 128 to both (no carry crosses between the
// halves, and a carry out of a half would only reach byte 2, which is not
// read here): six instructions where four adds and six byte selects were ten.
__device__ __forceinline__ void pack_low_digits(const uint32_t* w, uint32_t* pc, uint32_t* pb) {
  const uint32_t l01 = __builtin_amdgcn_perm(w[1], w[0], 0x05040100u);  // w0.lo16 | w1.lo16 << 16
  const uint32_t l23 = __builtin_amdgcn_perm(w[3], w[2], 0x05040100u);
  *pc = __builtin_amdgcn_perm(l23, l01, 0x06040200u);  // bytes 0 and 2 of each pair
  const u16x2 k = {128, 128};
  const uint32_t m01 = __builtin_bit_cast(uint32_t, __builtin_bit_cast(u16x2, l01) + k);
  const uint32_t m23 = __builtin_bit_cast(uint32_t, __builtin_bit_cast(u16x2, l23) + k);
  *pb = __builtin_amdgcn_perm(m23, m01, 0x07050301u);  // bytes 1 and 3 of each pair
}

// Bytes `byte` of four 32-bit words, packed low to high.
__device__ __forceinline__ uint32_t pack_bytes(uint32_t w0, uint32_t w1, uint32_t w2, uint32_t w3,
                                               uint32_t byte) {
  const uint32_t sel = 0x0c0c0400u | (byte * 0x0101u);  // [s1.byte, s0.byte, 0, 0]
  const uint32_t lo = __builtin_amdgcn_perm(w1, w0, sel);
  const uint32_t hi = __builtin_amdgcn_perm(w3, w2, sel);
  return __builtin_amdgcn_perm(hi, lo, 0x05040100u);
}

// Y = X - x_ref for producer wave pw's rows (rows at or beyond n are 0),
// quantized per row into the three digit planes of the stage buffer `lds`
// and the row's k (see above); with NEXT, as each row is written the load of
// that row for the full stage `next` is issued into its registers, and the
// reference row's last.
template <int NB, bool PAD, bool NEXT, class Src>
__device__ __forceinline__ void gram_put(uint8_t* __restrict__ lds, int n, int pw, int lane,
                                         f4* v, f4& vr, int ref, const StageRef<Src>& next) {
  const int wave = pw;
  const int64_t cn = next.c0 + 4 * lane;
  using S = GramShape<NB>;
  constexpr int P = S::RPW <= 4 ? 4 : (S::RPW <= 8 ? 8 : 16);
  constexpr int LB = P == 4 ? 2 : (P == 8 ? 3 : 4);
  int* kexp = reinterpret_cast<int*>(lds + 3 * S::PLANE);
  uint32_t m[P];
#pragma unroll
  for (int i = 0; i < P; ++i) m[i] = 0u;
#pragma unroll
  for (int i = 0; i < S::RPW; ++i) {
    const int row = wave * S::RPW + i;  // wave-uniform
    v[i] = v[i] - vr;
    if (PAD && row >= n) v[i] = f4{0.0f, 0.0f, 0.0f, 0.0f};
    const float a = __builtin_fmaxf(__builtin_fmaxf(__builtin_fabsf(v[i].x), __builtin_fabsf(v[i].y)),
                                    __builtin_fmaxf(__builtin_fabsf(v[i].z), __builtin_fabsf(v[i].w)));
    m[i] = __builtin_bit_cast(uint32_t, a);
  }
  // lane l: the largest |y| of row rho(l) of this wave; its exponent field e8
  // gives k = min(21 - E, 127) = 148 - max(e8, 21), E = max(e8, 1) - 127
  const uint32_t mx = transpose_max<P>(m, lane);
  const int e8 = static_cast<int>(mx >> 23);
  const int kl = 148 - (e8 > 21 ? e8 : 21);
  const int mine = bit_reverse(lane & (P - 1), LB);
  if (lane < P && mine < S::RPW) kexp[wave * S::RPW + mine] = kl;
#pragma unroll
  for (int i = 0; i < S::RPW; ++i) {
    const int row = wave * S::RPW + i;
    const int k = __builtin_amdgcn_readlane(kl, bit_reverse(i, LB));
    const float scale = __builtin_bit_cast(float, static_cast<uint32_t>(k + 127) << 23);
    uint32_t w[4];
    w[0] = __builtin_bit_cast(uint32_t, __builtin_fmaf(v[i].x, scale, kRoundMagic));
    w[1] = __builtin_bit_cast(uint32_t, __builtin_fmaf(v[i].y, scale, kRoundMagic));
    w[2] = __builtin_bit_cast(uint32_t, __builtin_fmaf(v[i].z, scale, kRoundMagic));
    w[3] = __builtin_bit_cast(uint32_t, __builtin_fmaf(v[i].w, scale, kRoundMagic));
    // the low 22 bits of w are those of q (w = bits(1.5 * 2^23 + q)); the
    // constant's bit 22 is taken out where the third byte is read
    uint32_t pc, pb;
    pack_low_digits(w, &pc, &pb);
    constexpr uint32_t kA = 32896u - 4194304u;  // + 32896, minus the constant's 2^22
    const uint32_t pa = pack_bytes(w[0] + kA, w[1] + kA, w[2] + kA, w[3] + kA, 2);
    const int off = row * kPlanePitch + 4 * lane;
    *reinterpret_cast<uint32_t*>(lds + off) = pa;
    *reinterpret_cast<uint32_t*>(lds + S::PLANE + off) = pb;
    *reinterpret_cast<uint32_t*>(lds + 2 * S::PLANE + off) = pc;
    if constexpr (NEXT) v[i] = gram_load<true>(next.src, load_row<PAD>(row, n, ref), cn, next.d);
  }
  if constexpr (NEXT) vr = gram_load<true>(next.src, ref, cn, next.d);
}

__device__ __forceinline__ i4 mfma_i8(const i4& a, const i4& b, const i4& c) {
  return __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, c, 0, 0, 0);
}

// The nine digit products of block pair q = CV + 4P of consumer wave CV
// (and of its later pairs, by recursion: every pair's blocks, and with them
// its fragment registers, are compile-time constants).
template <int NB, int CV, int P>
__device__ __forceinline__ void gram_pair_mfma(const i4* fa, const i4* fb, const i4* fc,
                                               i4 (*acc)[5]) {
  using S = GramShape<NB>;
  constexpr int q = CV + 4 * P;
  if constexpr (P < S::PPW && q < S::NBP) {
    constexpr int b1 = pair_b1(NB, q), b2 = pair_b2(NB, q);
    i4* A = acc[P];
    A[0] = mfma_i8(fa[b1], fa[b2], A[0]);
    A[1] = mfma_i8(fa[b1], fb[b2], A[1]);
    A[2] = mfma_i8(fa[b1], fc[b2], A[2]);
    A[1] = mfma_i8(fb[b1], fa[b2], A[1]);
    A[2] = mfma_i8(fb[b1], fb[b2], A[2]);
    A[3] = mfma_i8(fb[b1], fc[b2], A[3]);
    A[2] = mfma_i8(fc[b1], fa[b2], A[2]);
    A[3] = mfma_i8(fc[b1], fb[b2], A[3]);
    A[4] = mfma_i8(fc[b1], fc[b2], A[4]);
    gram_pair_mfma<NB, CV, P + 1>(fa, fb, fc, acc);
  }
}

// The exact stage value of each G entry of pair q = CV + 4P (and later
// pairs) added into acc64 (lane l, component e: row 16*b1 + 4*(l/16) + e,
// column 16*b2 + l%16).
template <int NB, int CV, int P>
__device__ __forceinline__ void gram_pair_flush(const int* kexp, int g, int r,
                                                const i4 (*acc)[5], double (*acc64)[4]) {
  using S = GramShape<NB>;
  constexpr int q = CV + 4 * P;
  if constexpr (P < S::PPW && q < S::NBP) {
    constexpr int b1 = pair_b1(NB, q), b2 = pair_b2(NB, q);
    const i4 kr = *reinterpret_cast<const i4*>(kexp + 16 * b1 + 4 * g);
    const int kc = kexp[16 * b2 + r];
    const i4* A = acc[P];
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      double t = static_cast<double>(A[0][e]);
      t = __builtin_fma(t, 256.0, static_cast<double>(A[1][e]));
      t = __builtin_fma(t, 256.0, static_cast<double>(A[2][e]));
      t = __builtin_fma(t, 256.0, static_cast<double>(A[3][e]));
      t = __builtin_fma(t, 256.0, static_cast<double>(A[4][e]));
      acc64[P][e] += __builtin_ldexp(t, -(kr[e] + kc));
    }
    gram_pair_flush<NB, CV, P + 1>(kexp, g, r, acc, acc64);
  }
}

// Consumer wave CV's block pairs over the stage in the buffer `lds`: the
// nine digit products of each pair into its five weight accumulators, chunk
// by chunk, then the stage's exact G entries added into acc64.
template <int NB, int CV>
__device__ __forceinline__ void gram_multiply(const uint8_t* __restrict__ lds, int g, int r,
                                              double (*acc64)[4]) {
  using S = GramShape<NB>;
  const int* kexp = reinterpret_cast<const int*>(lds + 3 * S::PLANE);
  i4 acc[S::PPW][5];
  const i4 zero = i4{0, 0, 0, 0};
#pragma unroll
  for (int p = 0; p < S::PPW; ++p)
#pragma unroll
    for (int t = 0; t < 5; ++t) acc[p][t] = zero;
#pragma unroll
  for (int ch = 0; ch < kGramStage / 64; ++ch) {
    i4 fa[NB], fb[NB], fc[NB];  // digit fragments a, b, c of every block
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const int off = (16 * b + r) * kPlanePitch + 64 * ch + 16 * g;
      fa[b] = *reinterpret_cast<const i4*>(lds + off);
      fb[b] = *reinterpret_cast<const i4*>(lds + S::PLANE + off);
      fc[b] = *reinterpret_cast<const i4*>(lds + 2 * S::PLANE + off);
    }
    gram_pair_mfma<NB, CV, 0>(fa, fb, fc, acc);
  }
  gram_pair_flush<NB, CV, 0>(kexp, g, r, acc, acc64);
}

// Partials of a workgroup: entry q*256 + row*16 + col holds
// G[16*b1 + row][16*b2 + col]; consumer wave c holds pairs q = c, c + 4, ...
// (MFMA output: lane l, component e is row 4*(l/16) + e, column l%16).
// out[entry * stride].
template <int NB, int CV>
__device__ __forceinline__ void gram_write_partials(const double (*acc64)[4], int g, int r,
                                                    double* __restrict__ out, int64_t stride) {
  using S = GramShape<NB>;
#pragma unroll
  for (int p = 0; p < S::PPW; ++p) {
    const int q = CV + 4 * p;  // entries only: no register choice depends on q
    if (q < S::NBP) {
#pragma unroll
      for (int e = 0; e < 4; ++e) out[(q * 256 + (4 * g + e) * 16 + r) * stride] = acc64[p][e];
    }
  }
}

// A batch of segments for one Gram table launch (by value in the kernel
// arguments): ffirst[s] = full stages before segment s (ffirst[count] = all
// of them), pfirst[s] = partial stages before segment s (pfirst[count] = all
// of them), and each segment's length.
struct GramSegs {
  int count;
  int32_t ffirst[kSegMax + 1];
  int32_t pfirst[kSegMax + 1];
  int64_t dims[kSegMax];
};

// The schedule of a workgroup. Its stages are entries s, s + G, ... (s its
// slot) of a list that holds every full stage first and then the partial
// ones (G = grid size, one workgroup per CU), `cnt` entries of which the
// first `nf` are full. In iteration i the producers quantize entry i into
// buffer i % 2 and the consumers multiply entry i - 1 from buffer
// (i - 1) % 2; a barrier ends every iteration. Iterations run DEPTH at a
// time while all those entries are full stages, with every load
// unconditional (so the compiler keeps the next DEPTH stages' loads in
// flight across the quantizing); the rest (the full stages past the last
// multiple of DEPTH, the partial stages and the final multiply) go one at a
// time with guarded loads.

// Consumer wave CV, then its partials.
template <int NB, int CV>
__device__ __forceinline__ void gram_consume(const uint8_t* __restrict__ lds, int64_t cnt,
                                             int64_t nf, double* __restrict__ out,
                                             int64_t stride) {
  using S = GramShape<NB>;
  const int lane = threadIdx.x & 63;
  const int g = lane >> 4, r = lane & 15;
  double acc64[S::PPW][4];
#pragma unroll
  for (int i = 0; i < S::PPW; ++i)
#pragma unroll
    for (int e = 0; e < 4; ++e) acc64[i][e] = 0.0;
  constexpr int D = S::DEPTH;
  int64_t t = 0;
  if (nf >= D) {
    for (; t + D - 1 < nf; t += D) {
#pragma unroll
      for (int u = 0; u < D; ++u) {  // iteration t + u: entry t + u - 1, buffer (t + u + 1) % 2
        if (u > 0 || t >= 1)
          gram_multiply<NB, CV>(lds + ((t + u + 1) & 1) * S::BUF, g, r, acc64);
        lds_barrier();
      }
    }
  }
  for (int64_t i = t; i <= cnt; ++i) {
    if (i >= 1) gram_multiply<NB, CV>(lds + ((i - 1) & 1) * S::BUF, g, r, acc64);
    lds_barrier();
  }
  gram_write_partials<NB, CV>(acc64, g, r, out, stride);
}

// Producer wave pw. `list.entry(i)` is this workgroup's i-th stage.
template <int NB, bool PAD, class List>
__device__ __forceinline__ void gram_produce(uint8_t* __restrict__ lds, int64_t cnt, int64_t nf,
                                             int n, int ref, int pw, const List& list) {
  using S = GramShape<NB>;
  const int lane = threadIdx.x & 63;
  constexpr int D = S::DEPTH;
  f4 v[D][S::RPW];
  f4 vr[D];
  int64_t t = 0;
  if (nf >= D) {
    // D stages in flight, one register set each; entries past the last full
    // one load that one again (not used)
    auto whole = [&](int64_t i) { return list.entry(i < nf ? i : nf - 1); };
#pragma unroll
    for (int u = 0; u < D; ++u) gram_issue<NB, PAD, true>(whole(u), n, ref, pw, lane, v[u], vr[u]);
    for (; t + D - 1 < nf; t += D) {
#pragma unroll
      for (int u = 0; u < D; ++u) {  // iteration t + u: buffer (t + u) % 2
        gram_put<NB, PAD, true>(lds + ((t + u) & 1) * S::BUF, n, pw, lane, v[u], vr[u], ref,
                                whole(t + u + D));
        lds_barrier();
      }
    }
  }
  for (int64_t i = t; i <= cnt; ++i) {
    if (i < cnt) {
      const auto st = list.entry(i);
      gram_issue<NB, PAD, false>(st, n, ref, pw, lane, v[0], vr[0]);
      gram_put<NB, PAD, false>(lds + (i & 1) * S::BUF, n, pw, lane, v[0], vr[0], ref, st);
    }
    lds_barrier();
  }
}

template <int NB, bool PAD, class List>
__device__ __forceinline__ void gram_run(uint8_t* __restrict__ lds, int64_t cnt, int64_t nf,
                                         int n, int ref, const List& list,
                                         double* __restrict__ out, int64_t stride) {
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave-uniform
  // the roles are compile-time per wave, so that every consumer's block
  // pairs, and with them its fragment registers, are constants
  switch (wave - kGramProducers) {
    case 0: gram_consume<NB, 0>(lds, cnt, nf, out, stride); break;
    case 1: gram_consume<NB, 1>(lds, cnt, nf, out, stride); break;
    case 2: gram_consume<NB, 2>(lds, cnt, nf, out, stride); break;
    case 3: gram_consume<NB, 3>(lds, cnt, nf, out, stride); break;
    default: gram_produce<NB, PAD>(lds, cnt, nf, n, ref, wave, list); break;
  }
}

// The workgroup's slot among the G of a launch: list entry slot + i * G is
// its i-th stage. Workgroups are dealt to the 8 XCDs round-robin (block b to
// XCD b % 8), so slot (b % 8) * (G / 8) + b / 8 gives each XCD a contiguous
// run of slots, and stages next to each other, which share the cache lines
// at the ends of their 1 KB row runs, meet in one XCD's L2 at about the same
// time instead of being fetched by two XCDs. (A bijection on [0, G) when 8
// divides G; other grids keep b.)
__device__ __forceinline__ int64_t gram_slot() {
  const int64_t b = blockIdx.x, G = gridDim.x;
  if (G % 8 != 0) return b;
  return (b % 8) * (G / 8) + b / 8;
}

// Entries of this workgroup's slot b among `total` list entries of which the
// first `nfull` are full stages: (count, full count).
__device__ __forceinline__ void gram_share(int64_t total, int64_t nfull, int64_t* cnt,
                                           int64_t* nf) {
  const int64_t b = gram_slot(), G = gridDim.x;
  *cnt = total > b ? (total - b + G - 1) / G : 0;
  *nf = nfull > b ? (nfull - b + G - 1) / G : 0;
}

// The stages of an n x d matrix: full stage s at coordinate 256 s, then the
// partial last one (when 256 does not divide d).
struct MatrixStages {
  const float* x;
  int64_t d;
  int64_t nfull;
  __device__ __forceinline__ StageRef<MatrixRows> entry(int64_t i) const {
    const int64_t li = gram_slot() + i * gridDim.x;  // list index (the partial stage is last)
    return StageRef<MatrixRows>{MatrixRows{x, d}, li * kGramStage, d, li < nfull};
  }
};

template <int NB, bool PAD>
__global__ __launch_bounds__(kGramThreads) __attribute__((amdgpu_waves_per_eu(kGramWavesPerSimd)))
void k_dist_gram(const float* __restrict__ x, int n, int64_t d,
                 const int32_t* __restrict__ ref_idx, double* __restrict__ partial) {
  using S = GramShape<NB>;
  __shared__ __attribute__((aligned(16))) uint8_t lds[S::LDS];
  const int ref = *ref_idx;
  const int64_t nfull = d / kGramStage;
  const int64_t total = (d + kGramStage - 1) / kGramStage;
  int64_t cnt, nf;
  gram_share(total, nfull, &cnt, &nf);
  gram_run<NB, PAD>(lds, cnt, nf, n, ref, MatrixStages{x, d, nfull}, partial + blockIdx.x,
                    gridDim.x);
}

// ---------------------------------------------------------------------------
// The Gram engine over a table of segments (segment s of vector i at
// ptrs[s * n + i], dims[s] floats). The list of a launch holds the full
// stages of all its segments in segment order (segment s owns list entries
// ffirst[s] .. ffirst[s+1]-1), then the partial last stage of every segment
// whose length 256 does not divide (entries nfull + pfirst[s] for those),
// and the workgroup of slot s takes entries s, s + G, ..., each with its
// segment's rows.
// One reference row index serves every segment (D is the same whatever row
// each coordinate is shifted by). Tile b of the launch writes column
// tile_base + b of partials with `tiles` columns in all.
__device__ __forceinline__ int last_le(const int32_t* first, int count, int64_t v) {
  int lo = 0, hi = count - 1;  // the last s with first[s] <= v
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (first[mid] <= v) lo = mid;
    else hi = mid - 1;
  }
  return lo;
}

struct TableStages {
  const float* const* ptrs;
  int n;
  const GramSegs* segs;
  __device__ __forceinline__ StageRef<TableRows> entry(int64_t i) const {
    const GramSegs& t = *segs;
    const int64_t li = gram_slot() + i * gridDim.x;
    const int64_t nfull = t.ffirst[t.count];
    if (li < nfull) {
      const int sg = last_le(t.ffirst, t.count, li);
      return StageRef<TableRows>{TableRows{ptrs + static_cast<int64_t>(sg) * n},
                                 (li - t.ffirst[sg]) * kGramStage, t.dims[sg], true};
    }
    // the partial stages: segment sg is the last with pfirst[sg] <= j (and
    // has one, since pfirst grows exactly at the segments that have one)
    const int sg = last_le(t.pfirst, t.count, li - nfull);
    const int64_t c0 = (t.dims[sg] / kGramStage) * kGramStage;
    return StageRef<TableRows>{TableRows{ptrs + static_cast<int64_t>(sg) * n}, c0, t.dims[sg],
                               false};
  }
};

template <int NB, bool PAD>
__global__ __launch_bounds__(kGramThreads) __attribute__((amdgpu_waves_per_eu(kGramWavesPerSimd)))
void k_dist_gram_table(const float* const* __restrict__ ptrs, GramSegs segs, int n,
                       const int32_t* __restrict__ ref_idx, int64_t tile_base, int64_t tiles,
                       double* __restrict__ partial) {
  using S = GramShape<NB>;
  __shared__ __attribute__((aligned(16))) uint8_t lds[S::LDS];
  const int ref = *ref_idx;
  const int64_t nfull = segs.ffirst[segs.count];
  const int64_t total = nfull + segs.pfirst[segs.count];
  int64_t cnt, nf;
  gram_share(total, nfull, &cnt, &nf);
  gram_run<NB, PAD>(lds, cnt, nf, n, ref, TableStages{ptrs, n, &segs},
                    partial + tile_base + blockIdx.x, tiles);
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
    launch("dist_gram", k_dist_gram<NB, true>, dim3(static_cast<unsigned>(p.tiles)), dim3(kGramThreads),
           0, s, x, p.n, p.d, ref, partial);
  else
    launch("dist_gram", k_dist_gram<NB, false>, dim3(static_cast<unsigned>(p.tiles)), dim3(kGramThreads),
           0, s, x, p.n, p.d, ref, partial);
  return hipGetLastError();
}

size_t align256(size_t b) { return (b + 255) & ~static_cast<size_t>(255); }

template <int NB>
int gram_blocks_per_cu_nb() {
  int blocks = 0, blocks_pad = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, k_dist_gram<NB, false>, kGramThreads, 0) !=
          hipSuccess ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks_pad, k_dist_gram<NB, true>, kGramThreads,
                                                   0) != hipSuccess ||
      blocks <= 0) {
    (void)hipGetLastError();
    return 1;
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
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, k_dist_gram_table<NB, false>, kGramThreads,
                                                   0) != hipSuccess ||
      hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks_pad, k_dist_gram_table<NB, true>,
                                                   kGramThreads, 0) != hipSuccess ||
      blocks <= 0) {
    (void)hipGetLastError();
    return 1;
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
    GramSegs tab{};
    tab.count = K - g0 < kSegMax ? K - g0 : kSegMax;
    int64_t full = 0, part = 0;
    for (int sg = 0; sg < tab.count; ++sg) {
      tab.ffirst[sg] = static_cast<int32_t>(full);
      tab.pfirst[sg] = static_cast<int32_t>(part);
      tab.dims[sg] = dims[g0 + sg];
      full += dims[g0 + sg] / kGramStage;
      part += dims[g0 + sg] % kGramStage != 0 ? 1 : 0;
      if (full + part > 0x7fffffff) return hipErrorInvalidValue;
    }
    tab.ffirst[tab.count] = static_cast<int32_t>(full);
    tab.pfirst[tab.count] = static_cast<int32_t>(part);
    const int64_t total = full + part;
    if (total == 0) continue;
    const hipError_t e = f(g0, tab, total < slots ? total : slots);
    if (e != hipSuccess) return e;
  }
  return hipSuccess;
}

template <int NB>
hipError_t launch_gram_table_nb(const float* const* ptrs, int n, const GramSegs& tab,
                                int64_t groups, const int32_t* ref, int64_t base, int64_t tiles,
                                double* partial, hipStream_t s) {
  if (n < 16 * NB)
    launch("dist_gram_table", k_dist_gram_table<NB, true>, dim3(static_cast<unsigned>(groups)),
           dim3(kGramThreads), 0, s, ptrs, tab, n, ref, base, tiles, partial);
  else
    launch("dist_gram_table", k_dist_gram_table<NB, false>, dim3(static_cast<unsigned>(groups)),
           dim3(kGramThreads), 0, s, ptrs, tab, n, ref, base, tiles, partial);
  return hipGetLastError();
}

int g_direct_max_n = 20;

}  // namespace

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

int64_t table_gram_tiles(const int64_t* dims, int K, int n) {
  int64_t tiles = 0;
  const hipError_t e = for_each_gram_launch(n, dims, K, [&](int, const GramSegs&, int64_t groups) {
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
  return for_each_gram_launch(n, dims, K, [&](int g0, const GramSegs& tab, int64_t groups) {
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

int load_width(const float* p) { return reinterpret_cast<uintptr_t>(p) % 4 == 0 ? 4 : 1; }

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
    p.width = load_width(x);
    if (p.width > direct_width_cap(n)) p.width = direct_width_cap(n);
    p.chunk = direct_chunk(d, p.width);
    p.entries = n * (n - 1) / 2;
  } else {
    p.engine = kEngineGram;
    p.width = 4;  // 16-byte loads of 1 KB row runs
    // As many workgroups as the device holds resident (at most one per
    // stage); slot s takes stages s, s + tiles, ... (the partial last stage,
    // if any, among them).
    const int nb = (n + 15) / 16;
    const int64_t slots = static_cast<int64_t>(device_cus()) * gram_blocks_per_cu(nb);
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
