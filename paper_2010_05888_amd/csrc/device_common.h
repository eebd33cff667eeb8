// Device-side helpers shared by the libgarfield kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace garfield {

typedef float f2 __attribute__((ext_vector_type(2)));
typedef float f4 __attribute__((ext_vector_type(4)));
// The same vectors at the alignment of a float: global memory on CDNA serves
// 8- and 16-byte accesses at any dword-aligned address, so rows of any length
// d stream with 16-byte loads (row i starts at i * d floats, which is 16-byte
// aligned only when d % 4 == 0).
typedef float f2u __attribute__((ext_vector_type(2), aligned(4)));
typedef float f4u __attribute__((ext_vector_type(4), aligned(4)));
// Two doubles (16-byte aligned).
typedef double d2 __attribute__((ext_vector_type(2)));

// min / max on finite values (inputs are finite by contract).
__device__ __forceinline__ float fmin_(float a, float b) { return __builtin_fminf(a, b); }
__device__ __forceinline__ float fmax_(float a, float b) { return __builtin_fmaxf(a, b); }

// Load W consecutive floats (W in {1, 2, 4}); p must be 4-byte aligned.
// NT: a streaming (nontemporal) load, for data read exactly once.
template <int W, bool NT = true>
__device__ __forceinline__ void load_w(const float* __restrict__ p, float* v) {
  if constexpr (W == 4) {
    const f4u* q = reinterpret_cast<const f4u*>(p);
    const f4u t = NT ? __builtin_nontemporal_load(q) : *q;
    v[0] = t.x; v[1] = t.y; v[2] = t.z; v[3] = t.w;
  } else if constexpr (W == 2) {
    const f2u* q = reinterpret_cast<const f2u*>(p);
    const f2u t = NT ? __builtin_nontemporal_load(q) : *q;
    v[0] = t.x; v[1] = t.y;
  } else {
    v[0] = NT ? __builtin_nontemporal_load(p) : *p;
  }
}

template <int W>
__device__ __forceinline__ void store_w(float* __restrict__ p, const float* v) {
  if constexpr (W == 4) {
    f4u t;
    t.x = v[0]; t.y = v[1]; t.z = v[2]; t.w = v[3];
    __builtin_nontemporal_store(t, reinterpret_cast<f4u*>(p));
  } else if constexpr (W == 2) {
    f2u t;
    t.x = v[0]; t.y = v[1];
    __builtin_nontemporal_store(t, reinterpret_cast<f2u*>(p));
  } else {
    __builtin_nontemporal_store(v[0], p);
  }
}

// Guarded load of W consecutive floats: elements at or beyond `limit`
// (relative to p) read as 0.
template <int W>
__device__ __forceinline__ void load_w_tail(const float* __restrict__ p, int64_t limit, float* v) {
#pragma unroll
  for (int e = 0; e < W; ++e) v[e] = (e < limit) ? p[e] : 0.0f;
}

// Lowest lane of the calling wave (all 64 lanes active) holding the smallest
// v, or 64 when every v is +inf; every lane receives it. With lane i owning
// index i this is the lowest (v, index). The minimum is the device library's
// wave reduction (cross-lane DPP moves), then one ballot of the lanes that
// hold it.
extern "C" __device__ __attribute__((const)) double __ockl_wfred_min_f64(double);

__device__ __forceinline__ int wave_argmin_lane(double v) {
  const double m = __ockl_wfred_min_f64(v);
  if (m == __builtin_inf()) return 64;
  return __builtin_ctzll(__ballot(v == m));
}

// Sum of v over the 64 lanes of the calling wave (all active), by an xor
// butterfly: every lane receives the same bits, and the grouping is fixed, so
// the result depends only on which lane holds which value.
__device__ __forceinline__ double wave_sum(double v) {
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) v += __shfl_xor(v, m, 64);
  return v;
}

}  // namespace garfield
