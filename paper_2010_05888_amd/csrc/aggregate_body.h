// Per-coordinate bodies of the streaming aggregation kernels, shared by the
// kernels over one row-major matrix (aggregate.hip) and the kernels over a
// table of segments (segtable.hip). Each body handles W consecutive
// coordinates c .. c+W-1 of a segment of length d and writes them to out + c;
// the rows come from a source (rows.h) and a row rule (AllRows, ListedRows)
// says which of them are used. NT: nontemporal loads (rows read once); kernels whose
// workgroups share rows read them with ordinary loads, which stay in L2.
#pragma once

#include "device_common.h"
#include "internal.h"
#include "rows.h"

namespace garfield {

#include "networks.inc"

// The rows a body reads, as a type, so that its loop over the rows has no
// branch: AllRows reads rows 0 .. k-1, ListedRows the listed ones. Kernels
// given an optional list come in both forms and the host picks one: a choice
// made per row made each row's load wait for the scalar load of its own
// index, where branch-free indices are fetched together ahead of the loads.
struct AllRows {
  __device__ __forceinline__ int64_t operator()(int t) const { return t; }
};

// An index outside [0, n) breaks a precondition; it reads row n - 1 rather
// than memory outside the input (one unsigned minimum, and the row offset is
// then an unsigned 32 x 64-bit product: few scalar instructions per row).
struct ListedRows {
  const int32_t* list;
  int n;
  __device__ __forceinline__ int64_t operator()(int t) const {
    const uint32_t r = static_cast<uint32_t>(list[t]);
    const uint32_t last = static_cast<uint32_t>(n - 1);
    return static_cast<int64_t>(r < last ? r : last);
  }
};

// Row t of an optional list (rows 0 .. k-1 without one), by ListedRows' rule;
// for code outside the gathers' loops (staging, masks).
__device__ __forceinline__ int64_t row_of(const int32_t* __restrict__ rows, int t, int n) {
  return rows ? ListedRows{rows, n}(t) : static_cast<int64_t>(t);
}

template <int W>
__device__ __forceinline__ void store_out(float* __restrict__ out, int64_t c, int64_t d,
                                          bool full, const float* o) {
  if (full) {
    store_w<W>(out + c, o);
  } else {
    for (int e = 0; e < W && c + e < d; ++e) out[c + e] = o[e];
  }
}

// ---------------------------------------------------------------------------
// Mean of k rows: fp64 sum of the rows in the order listed, eight loads in
// flight at a time, one rounding at the end.
template <int W, bool FULL, bool NT, class Src, class L>
__device__ __forceinline__ void sum_rows_at(const Src& src, int64_t d, const L& rows, int k,
                                            int64_t c, double* acc) {
  int t = 0;
  for (; t + 8 <= k; t += 8) {
    float v[8][W];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const float* p = src.row(rows(t + u)) + c;
      if constexpr (FULL) load_w<W, NT>(p, v[u]); else load_w_tail<W>(p, d - c, v[u]);
    }
#pragma unroll
    for (int u = 0; u < 8; ++u)
#pragma unroll
      for (int e = 0; e < W; ++e) acc[e] += static_cast<double>(v[u][e]);
  }
  for (; t < k; ++t) {
    float v[W];
    const float* p = src.row(rows(t)) + c;
    if constexpr (FULL) load_w<W, NT>(p, v); else load_w_tail<W>(p, d - c, v);
#pragma unroll
    for (int e = 0; e < W; ++e) acc[e] += static_cast<double>(v[e]);
  }
}

template <int W, bool NT = true, class Src, class L>
__device__ __forceinline__ void mean_at(const Src& src, int64_t d, const L& rows, int k,
                                        int64_t c, float* __restrict__ out) {
  double acc[W];
#pragma unroll
  for (int e = 0; e < W; ++e) acc[e] = 0.0;
  const bool full = c + W <= d;
  if (full) sum_rows_at<W, true, NT>(src, d, rows, k, c, acc);
  else sum_rows_at<W, false, NT>(src, d, rows, k, c, acc);
  const double count = static_cast<double>(k);
  float o[W];
#pragma unroll
  for (int e = 0; e < W; ++e) o[e] = static_cast<float>(acc[e] / count);
  store_out<W>(out, c, d, full, o);
}

// ---------------------------------------------------------------------------
// Coordinate-wise median of K rows: all K loads back to back, then the
// selection network per coordinate.
template <int K, int W, bool NT = true, class Src, class L>
__device__ __forceinline__ void median_at(const Src& src, int64_t d, const L& rows, int64_t c,
                                          float* __restrict__ out) {
  using Net = MedianNet<K>;
  float v[K][W];
  const bool full = c + W <= d;
  if (full) {
#pragma unroll
    for (int t = 0; t < K; ++t) load_w<W, NT>(src.row(rows(t)) + c, v[t]);
  } else {
#pragma unroll
    for (int t = 0; t < K; ++t) load_w_tail<W>(src.row(rows(t)) + c, d - c, v[t]);
  }
  float o[W];
#pragma unroll
  for (int e = 0; e < W; ++e) {
    float a[K];
#pragma unroll
    for (int t = 0; t < K; ++t) a[t] = v[t][e];
    Net::run(a);
    if constexpr (K % 2 == 1) {
      o[e] = a[Net::LO];
    } else {  // mean of the two middle values, exact in fp64, rounded once
      o[e] = static_cast<float>((static_cast<double>(a[Net::LO]) +
                                 static_cast<double>(a[Net::HI])) * 0.5);
    }
  }
  store_out<W>(out, c, d, full, o);
}

// ---------------------------------------------------------------------------
// Bulyan with beta = 3 (theta = 2f + 3, the smallest n for f, so T is odd):
// only the ranks c-2 .. c+2 around the median s[c] can be taken, so a band
// network (BandNet) leaves them in registers and the rule below -- the same
// comparisons and the same fp64 sum as bulyan_at's general path -- runs on
// compile-time registers, without the LDS column.
template <int T>
__device__ __forceinline__ float bulyan3_of_band(const float* a) {
  using B = BandNet<T>;
  constexpr int c = (T - 1) / 2;  // n_left = n_right = c
  const double med = static_cast<double>(a[B::reg(c)]);
  auto take = [&](float lv, float rv) {  // L before R in the merge by (|v - med|, v)
    const double dl = med - static_cast<double>(lv);
    const double dr = static_cast<double>(rv) - med;
    return (dl < dr) || (dl == dr && lv < rv);
  };
  double sum = 0.0;
  if constexpr (T == 3) {  // the whole set
    sum += static_cast<double>(a[B::reg(0)]);
    sum += static_cast<double>(a[B::reg(1)]);
    sum += static_cast<double>(a[B::reg(2)]);
  } else {
    // L_1 = s[c-1] against R_2 = s[c+2], then L_2 = s[c-2] against R_1 = s[c+1]
    int a_taken = 0;
    if (take(a[B::reg(c - 1)], a[B::reg(c + 2)])) {
      a_taken = 1;
      if (take(a[B::reg(c - 2)], a[B::reg(c + 1)])) a_taken = 2;
    }
    const float x0 = a_taken == 0 ? a[B::reg(c)] : (a_taken == 1 ? a[B::reg(c - 1)] : a[B::reg(c - 2)]);
    const float x1 = a_taken == 0 ? a[B::reg(c + 1)] : (a_taken == 1 ? a[B::reg(c)] : a[B::reg(c - 1)]);
    const float x2 = a_taken == 0 ? a[B::reg(c + 2)] : (a_taken == 1 ? a[B::reg(c + 1)] : a[B::reg(c)]);
    sum += static_cast<double>(x0);
    sum += static_cast<double>(x1);
    sum += static_cast<double>(x2);
  }
  return static_cast<float>(sum / 3.0);
}

// ---------------------------------------------------------------------------
// Bulyan aggregation for theta = T selected rows, beta = T - 2f closest.
//
// With s[0..T-1] sorted: odd T has the median s[c], c = (T-1)/2, always kept,
// and K = beta-1 more to take; even T has med = (s[c-1]+s[c])/2, c = T/2, and
// K = beta to take. Left candidates L_a = s[c-a] (a = 1, 2, ...) and right
// candidates R_b (s[c+b] for odd T, s[c-1+b] for even T) are each ordered by
// increasing key, so the K taken are the first K of their merge: L_a is taken
// iff key(L_a) < key(R_{K+1-a}) (a missing R counts as +inf). The number of
// left values taken is the count of such a. `col` is this thread's column of
// a T x kBlock LDS array (col[r * kBlock]).
template <int T, int W, bool NT = true, class Src, class L>
__device__ __forceinline__ void bulyan_at(const Src& src, int64_t d, const L& sel, int beta,
                                          int64_t cc, float* col, float* __restrict__ out) {
  using Net = SortNet<T>;
  constexpr bool kOdd = (T % 2) == 1;
  constexpr int c = kOdd ? (T - 1) / 2 : T / 2;
  constexpr int n_left = c;                          // L_a exists for a <= n_left
  constexpr int n_right = kOdd ? T - 1 - c : T - c;  // R_b exists for b <= n_right
  const int K = kOdd ? beta - 1 : beta;
  float v[T][W];
  const bool full = cc + W <= d;
  if (full) {
#pragma unroll
    for (int t = 0; t < T; ++t) load_w<W, NT>(src.row(sel(t)) + cc, v[t]);
  } else {
#pragma unroll
    for (int t = 0; t < T; ++t) load_w_tail<W>(src.row(sel(t)) + cc, d - cc, v[t]);
  }
  float o[W];
  if constexpr (kOdd && T >= 3) {
    if (beta == 3) {  // uniform: the band network and registers only
#pragma unroll
      for (int e = 0; e < W; ++e) {
        float a[T];
#pragma unroll
        for (int t = 0; t < T; ++t) a[t] = v[t][e];
        BandNet<T>::run(a);
        o[e] = bulyan3_of_band<T>(a);
      }
      store_out<W>(out, cc, d, full, o);
      return;
    }
  }
#pragma unroll
  for (int e = 0; e < W; ++e) {
    float a[T];
#pragma unroll
    for (int t = 0; t < T; ++t) a[t] = v[t][e];
    Net::run(a);
#pragma unroll
    for (int r = 0; r < T; ++r) col[r * kBlock] = a[Net::reg(r)];
    const double med = kOdd ? static_cast<double>(col[c * kBlock])
                            : (static_cast<double>(col[(c - 1) * kBlock]) +
                               static_cast<double>(col[c * kBlock])) * 0.5;
    int a_taken = 0;
    for (int i = 1; i <= K; ++i) {
      if (i > n_left) break;
      const int b = K + 1 - i;
      bool take = true;
      if (b <= n_right) {
        const float lv = col[(c - i) * kBlock];
        const float rv = col[(kOdd ? c + b : c - 1 + b) * kBlock];
        const double dl = med - static_cast<double>(lv);
        const double dr = static_cast<double>(rv) - med;
        take = (dl < dr) || (dl == dr && lv < rv);
      }
      if (!take) break;
      a_taken = i;
    }
    const int lo = c - a_taken;
    const int hi = lo + beta - 1;  // inclusive
    double sum = 0.0;
    for (int r = lo; r <= hi; ++r) sum += static_cast<double>(col[r * kBlock]);
    o[e] = static_cast<float>(sum / static_cast<double>(beta));
  }
  store_out<W>(out, cc, d, full, o);
}

}  // namespace garfield
