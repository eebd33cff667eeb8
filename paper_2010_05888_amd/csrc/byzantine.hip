// Byzantine behaviour and the variance condition, on the device.
//
//  * Attacks. Garfield's Byzantine worker and server objects send reversed
//    vectors, random vectors, "little is enough" vectors and "fall of
//    empires" vectors (Section 3.2, Main objects); the Byzantine-behaviour
//    experiment uses random vectors and vectors reversed and amplified by -100
//    (Section 6.5). The kernels below write such rows from the honest ones, so
//    that a rule's input can be built in HBM without a host round trip.
//  * Variance condition (Section 3.1, Tradeoffs): a rule is safe when
//    kappa * Delta * sqrt(E||g - E g||^2) <= ||grad L|| for some kappa > 1.
//    The variance of the honest gradients is estimated from their pairwise
//    distances, since sum_i ||g_i - mean||^2 = (1/h) sum_{i<j} ||g_i - g_j||^2:
//    the distance step the rules already use gives it with no extra pass.

#include "device_common.h"
#include "dist_layout.h"
#include "internal.h"
#include "timing.h"

namespace garfield {

namespace {

// One workgroup per kBlock items (a single pass over d).
int blocks_for(int64_t items) {
  int64_t b = (items + kBlock - 1) / kBlock;
  if (b > 0x7fffffff) b = 0x7fffffff;
  return b < 1 ? 1 : static_cast<int>(b);
}

// ---------------------------------------------------------------------------
// Random vectors: Philox4x32-10 (Salmon, Moraes, Dror and Shaw, "Parallel
// random numbers: as easy as 1, 2, 3", SC'11), a counter-based generator:
// ten rounds, each multiplying two of the four counter words by fixed odd
// constants and mixing the high halves with the other words and the key,
// which is bumped by two Weyl constants between rounds. Counter (q_lo, q_hi,
// row, 0) with q = c / 4, key = the 64-bit seed: coordinate c of Byzantine row
// b depends only on (seed, b, c), never on the launch.
struct Words {
  uint32_t w[4];
};

__device__ __forceinline__ Words philox4x32_10(uint32_t c0, uint32_t c1, uint32_t c2, uint32_t c3,
                                                uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r > 0) {
      k0 += 0x9E3779B9u;
      k1 += 0xBB67AE85u;
    }
    const uint64_t p0 = static_cast<uint64_t>(0xD2511F53u) * c0;
    const uint64_t p1 = static_cast<uint64_t>(0xCD9E8D57u) * c2;
    const uint32_t n0 = static_cast<uint32_t>(p1 >> 32) ^ c1 ^ k0;
    const uint32_t n2 = static_cast<uint32_t>(p0 >> 32) ^ c3 ^ k1;
    c1 = static_cast<uint32_t>(p1);
    c3 = static_cast<uint32_t>(p0);
    c0 = n0;
    c2 = n2;
  }
  return Words{{c0, c1, c2, c3}};
}

// A 32-bit word to a uniform in (0, 1): (top 23 bits + 1/2) * 2^-23, exact in
// fp32, never 0 or 1.
__device__ __forceinline__ float unit_open(uint32_t w) {
  return (static_cast<float>(w >> 9) + 0.5f) * 0x1p-23f;
}

// Box-Muller: words (a, b) -> r cos(2 pi u_b), r sin(2 pi u_b), r = sqrt(-2 ln u_a).
__device__ __forceinline__ void box_muller(uint32_t a, uint32_t b, float* z0, float* z1) {
  const float r = sqrtf(-2.0f * logf(unit_open(a)));
  float s, c;
  sincospif(2.0f * unit_open(b), &s, &c);
  *z0 = r * c;
  *z1 = r * s;
}

template <int W>
__global__ __launch_bounds__(kBlock) void k_attack_gaussian(int64_t d, float sigma, uint32_t k0,
                                                            uint32_t k1, float* __restrict__ byz) {
  const int b = blockIdx.y;
  const int64_t q = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;  // quad of coordinates
  const int64_t c = 4 * q;
  if (c >= d) return;
  const Words w = philox4x32_10(static_cast<uint32_t>(q), static_cast<uint32_t>(q >> 32),
                                static_cast<uint32_t>(b), 0u, k0, k1);
  float z[4];
  box_muller(w.w[0], w.w[1], &z[0], &z[1]);
  box_muller(w.w[2], w.w[3], &z[2], &z[3]);
#pragma unroll
  for (int e = 0; e < 4; ++e) z[e] *= sigma;
  float* __restrict__ row = byz + static_cast<int64_t>(b) * d;
  if (c + 4 <= d) {
    if constexpr (W == 4) {
      store_w<4>(row + c, z);
    } else {
#pragma unroll
      for (int e = 0; e < 4; ++e) row[c + e] = z[e];
    }
  } else {
    for (int e = 0; e < 4 && c + e < d; ++e) row[c + e] = z[e];
  }
}

// ---------------------------------------------------------------------------
// Per-coordinate moments of the h honest rows, then the same value written to
// every Byzantine row: "little is enough" (mean - z * std, population std) or
// "fall of empires" (-eps * mean). One pass in fp64 on values shifted by the
// first honest row (exact differences of fp32 values), which keeps the
// variance free of cancellation: mean = v0 + S1/h, var = (S2 - S1^2/h) / h.
enum MomentKind { kLittle = 0, kEmpire = 1 };

template <int W, int KIND>
__global__ __launch_bounds__(kBlock) void k_attack_moments(const float* __restrict__ x, int h,
                                                           int64_t d, double param, int nbyz,
                                                           float* __restrict__ byz) {
  constexpr int kChunk = 16;  // rows whose loads are issued back to back
  const int64_t c = (static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x) * W;
  if (c >= d) return;
  const bool full = c + W <= d;
  float v0[W];
  double s1[W], s2[W];
  if (full) load_w<W>(x + c, v0);
  else load_w_tail<W>(x + c, d - c, v0);
#pragma unroll
  for (int e = 0; e < W; ++e) s1[e] = s2[e] = 0.0;
  for (int t0 = 1; t0 < h; t0 += kChunk) {
    float v[kChunk][W];
#pragma unroll
    for (int i = 0; i < kChunk; ++i) {
      if (t0 + i < h) {  // uniform
        const float* p = x + static_cast<int64_t>(t0 + i) * d + c;
        if (full) load_w<W>(p, v[i]);
        else load_w_tail<W>(p, d - c, v[i]);
      }
    }
#pragma unroll
    for (int i = 0; i < kChunk; ++i) {
      if (t0 + i < h) {
#pragma unroll
        for (int e = 0; e < W; ++e) {
          const double dv = static_cast<double>(v[i][e]) - static_cast<double>(v0[e]);
          s1[e] += dv;
          s2[e] = fma(dv, dv, s2[e]);
        }
      }
    }
  }
  float o[W];
  const double inv_h = 1.0 / static_cast<double>(h);
#pragma unroll
  for (int e = 0; e < W; ++e) {
    const double mean = static_cast<double>(v0[e]) + s1[e] * inv_h;
    if constexpr (KIND == kLittle) {
      double var = (s2[e] - s1[e] * (s1[e] * inv_h)) * inv_h;
      var = var > 0.0 ? var : 0.0;
      o[e] = static_cast<float>(mean - param * sqrt(var));
    } else {
      o[e] = static_cast<float>(-param * mean);
    }
  }
  for (int b = 0; b < nbyz; ++b) {
    float* __restrict__ row = byz + static_cast<int64_t>(b) * d;
    if (full) store_w<W>(row + c, o);
    else
      for (int e = 0; e < W && c + e < d; ++e) row[c + e] = o[e];
  }
}

// Reversed (and amplified) vectors: Byzantine row b = param * honest row b % h,
// the product formed in fp64 and rounded once.
template <int W>
__global__ __launch_bounds__(kBlock) void k_attack_scale(const float* __restrict__ x, int h,
                                                         int64_t d, double param,
                                                         float* __restrict__ byz) {
  const int b = blockIdx.y;
  const int64_t c = (static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x) * W;
  if (c >= d) return;
  const float* __restrict__ src = x + static_cast<int64_t>(b % h) * d;
  float* __restrict__ dst = byz + static_cast<int64_t>(b) * d;
  float v[W];
  if (c + W <= d) {
    load_w<W>(src + c, v);
#pragma unroll
    for (int e = 0; e < W; ++e) v[e] = static_cast<float>(param * static_cast<double>(v[e]));
    store_w<W>(dst + c, v);
  } else {
    for (int64_t e = c; e < d; ++e) dst[e] = static_cast<float>(param * static_cast<double>(src[e]));
  }
}

// ---------------------------------------------------------------------------
// Variance condition. k_sqnorm_partials: per workgroup, sum of t_c^2 over its
// kSqnormSteps * kBlock * W coordinates (each square exact in fp64; a lane's
// steps are kBlock * W apart), reduced in a fixed tree. k_variance_finish (one
// workgroup): the partials in a fixed order, and sum_{i<j} D[i][j] over the h
// honest rows, row by row.
constexpr int kSqnormSteps = 8;

template <int W>
__global__ __launch_bounds__(kBlock) void k_sqnorm_partials(const float* __restrict__ t, int64_t d,
                                                            double* __restrict__ partial) {
  __shared__ double red[kBlock];
  const int64_t base = static_cast<int64_t>(blockIdx.x) * kSqnormSteps * kBlock * W +
                       static_cast<int64_t>(threadIdx.x) * W;
  float v[kSqnormSteps][W];
#pragma unroll
  for (int k = 0; k < kSqnormSteps; ++k) {  // loads back to back
    const int64_t c = base + static_cast<int64_t>(k) * kBlock * W;
    if (c + W <= d) load_w<W>(t + c, v[k]);
    else if (c < d) load_w_tail<W>(t + c, d - c, v[k]);
    else
      for (int e = 0; e < W; ++e) v[k][e] = 0.0f;
  }
  double a = 0.0;
#pragma unroll
  for (int k = 0; k < kSqnormSteps; ++k)
#pragma unroll
    for (int e = 0; e < W; ++e) a = fma(static_cast<double>(v[k][e]), static_cast<double>(v[k][e]), a);
  red[threadIdx.x] = a;
  __syncthreads();
  for (int s = kBlock / 2; s > 0; s >>= 1) {
    if (static_cast<int>(threadIdx.x) < s) red[threadIdx.x] += red[threadIdx.x + s];
    __syncthreads();
  }
  if (threadIdx.x == 0) partial[blockIdx.x] = red[0];
}

__global__ __launch_bounds__(kBlock) void k_variance_finish(DistSums ds, int h,
                                                            const double* __restrict__ partial,
                                                            int64_t parts,
                                                            double* __restrict__ stats) {
  __shared__ double red[kBlock];
  __shared__ double rows[kNmax];
  double a = 0.0;
  for (int64_t p = threadIdx.x; p < parts; p += kBlock) a += partial[p];
  red[threadIdx.x] = a;
  const int i = threadIdx.x;
  if (i < h) {  // row i: its distances to the rows after it, in order
    double r = 0.0;
    for (int j = i + 1; j < h; ++j) r += dist_entry(ds, i, j);
    rows[i] = r;
  }
  __syncthreads();
  for (int s = kBlock / 2; s > 0; s >>= 1) {
    if (i < s) red[i] += red[i + s];
    __syncthreads();
  }
  if (i == 0) {
    double total = 0.0;
    for (int r = 0; r < h; ++r) total += rows[r];
    stats[0] = total / (static_cast<double>(h) * static_cast<double>(h - 1));
    stats[1] = red[0];
  }
}

template <int W>
hipError_t launch_attack_moments(int kind, const float* x, int h, int64_t d, double param,
                                 int nbyz, float* byz, hipStream_t s) {
  const dim3 grid(blocks_for((d + W - 1) / W));
  if (kind == kLittle)
    launch("attack_little", k_attack_moments<W, kLittle>, grid, dim3(kBlock), 0, s, x, h, d, param,
           nbyz, byz);
  else
    launch("attack_empire", k_attack_moments<W, kEmpire>, grid, dim3(kBlock), 0, s, x, h, d, param,
           nbyz, byz);
  return hipGetLastError();
}

template <int W>
hipError_t launch_attack_scale(const float* x, int h, int64_t d, double param, int nbyz,
                               float* byz, hipStream_t s) {
  launch("attack_reverse", k_attack_scale<W>,
         dim3(blocks_for((d + W - 1) / W), static_cast<unsigned>(nbyz)), dim3(kBlock), 0, s, x, h,
         d, param, byz);
  return hipGetLastError();
}

}  // namespace

hipError_t enqueue_attack(int kind, const float* honest, int h, int64_t d, double param,
                          uint64_t seed, float* byz, int nbyz, hipStream_t s) {
  if (d == 0 || nbyz == 0) return hipSuccess;
  const bool wide = load_width(byz) == 4 && (honest == nullptr || load_width(honest) == 4);
  switch (kind) {
    case kAttackReverse:
      return wide ? launch_attack_scale<4>(honest, h, d, param, nbyz, byz, s)
                  : launch_attack_scale<1>(honest, h, d, param, nbyz, byz, s);
    case kAttackRandom: {
      const dim3 grid(blocks_for((d + 3) / 4), static_cast<unsigned>(nbyz));
      const uint32_t k0 = static_cast<uint32_t>(seed), k1 = static_cast<uint32_t>(seed >> 32);
      if (wide)
        launch("attack_random", k_attack_gaussian<4>, grid, dim3(kBlock), 0, s, d,
               static_cast<float>(param), k0, k1, byz);
      else
        launch("attack_random", k_attack_gaussian<1>, grid, dim3(kBlock), 0, s, d,
               static_cast<float>(param), k0, k1, byz);
      return hipGetLastError();
    }
    case kAttackLittle:
    case kAttackEmpire: {
      const int mk = kind == kAttackLittle ? kLittle : kEmpire;
      return wide ? launch_attack_moments<4>(mk, honest, h, d, param, nbyz, byz, s)
                  : launch_attack_moments<1>(mk, honest, h, d, param, nbyz, byz, s);
    }
    default:
      return hipErrorInvalidValue;
  }
}

int64_t sqnorm_parts(int64_t d, const float* t) {
  const int64_t per = static_cast<int64_t>(kSqnormSteps) * kBlock * load_width(t);
  return (d + per - 1) / per;
}

hipError_t enqueue_variance_stats(const DistSums& ds, int h, const float* grad, int64_t d,
                                  double* partial, double* stats, hipStream_t s) {
  const int64_t parts = d > 0 ? sqnorm_parts(d, grad) : 0;
  if (parts > 0) {
    if (load_width(grad) == 4)
      launch("sqnorm", k_sqnorm_partials<4>, dim3(static_cast<unsigned>(parts)), dim3(kBlock), 0,
             s, grad, d, partial);
    else
      launch("sqnorm", k_sqnorm_partials<1>, dim3(static_cast<unsigned>(parts)), dim3(kBlock), 0,
             s, grad, d, partial);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  launch("variance_finish", k_variance_finish, dim3(1), dim3(kBlock), 0, s, ds, h, partial, parts,
         stats);
  return hipGetLastError();
}

}  // namespace garfield
