// Selection on the distance matrix D (n x n fp64, n <= 64, built in LDS from
// the distance step's entry sums): Krum / Multi-Krum
// scores and top-m, Bulyan's iterated Krum, and MDA's subset search
// (Section 3.1 items 2-4). All of it runs on the device so the selected
// indices never round-trip through the host; every ranking breaks ties
// towards the lower index and every sum is added in a fixed order.

#include "device_common.h"
#include "direct_body.h"
#include "dist_layout.h"
#include "internal.h"
#include "timing.h"

namespace garfield {

namespace {

// order[i*n + r] = the j != i whose (D[i][j], j) has rank r in row i (and,
// if pos is given, pos[i*n + j] = r), for an n x n D in LDS. Scores then walk
// a row in ascending distance order, which is the order the distances are
// added in (so identical rows get bit-identical scores).
__device__ void rank_rows(const double* D, int n, unsigned char* order, unsigned char* pos) {
  for (int idx = threadIdx.x; idx < n * n; idx += blockDim.x) {
    const int i = idx / n, j = idx % n;
    if (i == j) continue;
    const double v = D[idx];
    const double* row = D + i * n;
    int rank = 0;
#pragma unroll 8
    for (int j2 = 0; j2 < n; ++j2) {  // no branch: eight reads in flight at a time
      const double w = row[j2];
      rank += (j2 != i) & ((w < v) | ((w == v) & (j2 < j)));
    }
    order[i * n + rank] = static_cast<unsigned char>(j);
    if (pos) pos[idx] = static_cast<unsigned char>(rank);
  }
  __syncthreads();
}

__device__ void load_and_rank(const DistSums& ds, double* D, unsigned char* order,
                              unsigned char* pos = nullptr) {
  load_dist(ds, D);
  rank_rows(D, ds.n, order, pos);
}

// Called by the 64 lanes of wave 0: write the selected local indices a < n
// (bit a of the lane-uniform mask) to sel, as global indices map[a] (a itself
// when map is null), in ascending order of the global index.
__device__ void write_selected(uint64_t mask, int n, const int32_t* map,
                               int32_t* __restrict__ sel) {
  const int a = threadIdx.x;
  if (a >= n || !((mask >> a) & 1)) return;
  int pos;
  if (!map) {
    pos = __popcll(mask & ((uint64_t{1} << a) - 1));
  } else {
    pos = 0;
    const int ga = map[a];
    for (uint64_t rest = mask; rest; rest &= rest - 1) pos += map[__builtin_ctzll(rest)] < ga;
  }
  sel[pos] = map ? map[a] : a;
}

// Multi-Krum on an n x n D in LDS: score(i) = sum of the k = n-f-2 smallest
// D[i][j], j != i; flag[i] = i is among the m lowest (score, i). All threads
// of the block take part. One wave sums a row: lane r holds the row's r-th
// smallest distance, and the lanes below k are added by the wave's butterfly,
// so rows with the same distances (in any order) get bit-identical scores.
__device__ void krum_flags(const double* D, const unsigned char* order, int n, int f, int m,
                           double* score, int* flag) {
  const int k = n - f - 2;  // 1 .. n-2 (n >= 2f+3)
  const int lane = threadIdx.x & 63;
  for (int i = threadIdx.x >> 6; i < n; i += blockDim.x >> 6) {
    const double v = lane < k ? D[i * n + order[i * n + lane]] : 0.0;
    const double s = wave_sum(v);
    if (lane == 0) score[i] = s;
  }
  __syncthreads();
  const int i = threadIdx.x;
  if (i < n) {
    const double si = score[i];
    int rank = 0;
#pragma unroll 8
    for (int j = 0; j < n; ++j) {
      const double w = score[j];
      rank += (w < si) | ((w == si) & (j < i));
    }
    flag[i] = rank < m;
  }
  __syncthreads();
}

// Multi-Krum: the m lowest (score, i) are selected.
// The single-workgroup selections run 16 waves: the distance loads and the
// rankings (independent LDS reads per entry) spread over four times as many
// lanes as a kBlock workgroup has.
constexpr int kSelectThreads = 1024;

__global__ __launch_bounds__(kSelectThreads) void k_krum_select(DistSums ds, int f, int m,
                                                        int32_t* __restrict__ sel) {
  const int n = ds.n;
  __shared__ double D[kNmax * kNmax];
  __shared__ unsigned char order[kNmax * kNmax];
  __shared__ double score[kNmax];
  __shared__ int flag[kNmax];
  load_and_rank(ds, D, order);
  krum_flags(D, order, n, f, m, score, flag);
  if (threadIdx.x >= 64) return;
  const uint64_t mask = __ballot(static_cast<int>(threadIdx.x) < n && flag[threadIdx.x]);
  write_selected(mask, n, nullptr, sel);
}

// ---------------------------------------------------------------------------
// Multi-Krum's selection and mean in one kernel, for short inputs (n <=
// kFusedMaxN rows, 16-byte loads) whose distance step left its tile partials
// folded: a launch and the full-size selection workgroup cost more than the
// work itself at such sizes. Every workgroup takes 1,024 coordinates: it loads
// them from all n rows first, adds the tiles while those loads are in flight,
// makes the selection in one wave, and writes the mean of the selected rows
// from its registers. Each step keeps the arithmetic of the separate kernels
// (load_dist's tile sums, krum_flags' scores and ranking, k_mean_rows' mean),
// so the selection and the output are bit-identical to theirs.

// The folded tile partials of all P entries (entry-major, `tiles` <= 256 per
// entry) summed into esum, every load issued before the first addition: wave
// w takes entries w, w + 4, ...; each sum is formed in the tile-sum kernel's
// order, exactly as load_dist forms it.
template <int P>
__device__ __forceinline__ void fold_tiles(const double* __restrict__ partial, int64_t tiles,
                                           double* esum) {
  constexpr int kWaves = kBlock / 64;
  constexpr int E = (P + kWaves - 1) / kWaves;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  // unconditional loads from clamped addresses (all in flight at once); the
  // values of slots past `tiles` are replaced by 0
  double v[E];
#pragma unroll
  for (int k = 0; k < E; ++k) {
    const int e = wave + k * kWaves;
    const double* row = partial + static_cast<int64_t>(e < P ? e : P - 1) * tiles;
    double s[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int t = lane + 64 * u;
      const double val = row[t < tiles ? t : 0];
      s[u] = t < tiles ? val : 0.0;
    }
    v[k] = (s[0] + s[2]) + (s[1] + s[3]);
  }
#pragma unroll
  for (int k = 0; k < E; ++k) {
    const int e = wave + k * kWaves;
    if (e < P) {
#pragma unroll
      for (int m = 32; m > 0; m >>= 1) v[k] += __shfl_xor(v[k], m, 64);
      if (lane == 0) esum[e] = v[k];
    }
  }
  __syncthreads();
}

// Multi-Krum's selection from the N x N distances (entry sums esum, direct
// layout), by the 64 lanes of one wave without LDS traffic or barriers: lane
// i < N sorts its row's N-1 distances, adds the k = N-f-2 smallest as the
// butterfly of krum_flags adds them (a balanced tree in ascending order, the
// other slots 0: the same bits), and ranks its (score, i) against every
// lane's. Returns the lane-uniform mask of the m selected rows.
template <int N>
__device__ __forceinline__ uint64_t krum_mask_wave(const double* esum, int f, int m) {
  constexpr int M = N - 1;
  const int i = threadIdx.x & 63;
  const int k = N - f - 2;
  double score = 0.0;
  if (i < N) {
    double r[M];
#pragma unroll
    for (int q = 0; q < M; ++q) {
      const int j = q < i ? q : q + 1;
      r[q] = esum[direct_entry(N, i < j ? i : j, i < j ? j : i)];
    }
#pragma unroll
    for (int a = 0; a < M; ++a)  // bubble network: ascending
#pragma unroll
      for (int b = 0; b + 1 < M - a; ++b) {
        const double lo = __builtin_fmin(r[b], r[b + 1]);
        r[b + 1] = __builtin_fmax(r[b], r[b + 1]);
        r[b] = lo;
      }
    double t[16];
#pragma unroll
    for (int q = 0; q < 16; ++q) t[q] = (q < M && q < k) ? r[q < M ? q : 0] : 0.0;
#pragma unroll
    for (int h = 1; h < 16; h <<= 1)
#pragma unroll
      for (int q = 0; q < 16; q += 2 * h) t[q] = t[q] + t[q + h];
    score = t[0];
  }
  const int64_t bits = __double_as_longlong(score);
  const int lo = static_cast<int>(bits), hi = static_cast<int>(bits >> 32);
  int rank = 0;
#pragma unroll
  for (int j = 0; j < N; ++j) {
    const uint64_t sj_bits =
        (static_cast<uint64_t>(static_cast<uint32_t>(__builtin_amdgcn_readlane(hi, j))) << 32) |
        static_cast<uint32_t>(__builtin_amdgcn_readlane(lo, j));
    const double sj = __longlong_as_double(static_cast<int64_t>(sj_bits));
    rank += (sj < score) | ((sj == score) & (j < i));
  }
  return __ballot(i < N && rank < m);
}

template <int N>
__global__ __launch_bounds__(kBlock) void k_krum_select_mean(const float* __restrict__ x,
                                                             int64_t d,
                                                             const double* __restrict__ partial,
                                                             int64_t tiles, int f, int m,
                                                             int32_t* __restrict__ sel,
                                                             float* __restrict__ out) {
  constexpr int W = 4, P = N * (N - 1) / 2;
  __shared__ double esum[P];
  __shared__ uint64_t mask_s;
  const int64_t c = (static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x) * W;
  float v[N][W];
  if (c < d) direct_load<N, W>(MatrixRows{x, d}, c, d, v);
  fold_tiles<P>(partial, tiles, esum);
  if (threadIdx.x < 64) {
    const uint64_t mask = krum_mask_wave<N>(esum, f, m);
    if (threadIdx.x == 0) mask_s = mask;
    if (blockIdx.x == 0) write_selected(mask, N, nullptr, sel);
  }
  __syncthreads();
  if (c >= d) return;
  const uint64_t mask = mask_s;
  double s[W] = {0.0, 0.0, 0.0, 0.0};
#pragma unroll
  for (int i = 0; i < N; ++i) {
    if ((mask >> i) & 1) {
#pragma unroll
      for (int e = 0; e < W; ++e) s[e] += static_cast<double>(v[i][e]);
    }
  }
  const double count = static_cast<double>(m);
  float o[W];
#pragma unroll
  for (int e = 0; e < W; ++e) o[e] = static_cast<float>(s[e] / count);
  if (c + W <= d) {
    store_w<W>(out + c, o);
  } else {
    for (int e = 0; e < W && c + e < d; ++e) out[c + e] = o[e];
  }
}

// Workgroups of k_krum_select_mean for d coordinates.
int64_t select_mean_groups(int64_t d) {
  const int64_t per = static_cast<int64_t>(kBlock) * 4;
  return (d + per - 1) / per;
}

template <int N>
hipError_t launch_select_mean(const float* x, int64_t d, const DistSums& ds, int f, int m,
                              int32_t* sel, float* out, hipStream_t s) {
  launch("krum_select_mean", k_krum_select_mean<N>, dim3(static_cast<unsigned>(select_mean_groups(d))),
         dim3(kBlock), 0, s, x, d, ds.partial, ds.tiles, f, m, sel, out);
  return hipGetLastError();
}

template <int N>
hipError_t select_mean_dispatch(int n, const float* x, int64_t d, const DistSums& ds, int f,
                                int m, int32_t* sel, float* out, hipStream_t s) {
  if constexpr (N > kFusedMaxN) {
    return hipErrorInvalidValue;
  } else {
    if (n == N) return launch_select_mean<N>(x, d, ds, f, m, sel, out, s);
    return select_mean_dispatch<N + 1>(n, x, d, ds, f, m, sel, out, s);
  }
}

// Iterated Krum, Bulyan's selection (theta = n-2f rounds) and the iterated
// Multi-Krum variant (m rounds): each round scores every remaining
// vector against the other remaining ones with k = max(r-f-2, 0) neighbours
// (r = vectors remaining) and moves the lowest (score, index) to the
// selection. Round 0 sums every row's k nearest in ascending order; after
// that a row's score follows the removals: when the pick p leaves and k drops
// by one, the new score is the old one minus D[i][p] if p was among i's k
// nearest, else minus the k-th nearest (tracked by its position in the
// row's ranking, which then steps back to the previous remaining vector); with
// one neighbour left the score is reset to that distance itself.
// After the ranking the rounds run in wave 0 alone (n <= 64: lane i owns row
// i), with the remaining set as a 64-bit mask every lane holds, so a round
// needs no workgroup barrier.
// Called by the 64 lanes of wave 0 on a ranked n x n D in LDS; returns the
// lane-uniform mask of the picked rows.
__device__ uint64_t krum_rounds_mask(const double* D, const unsigned char* order,
                                     const unsigned char* pos, int n, int f, int rounds) {
  const int i = threadIdx.x;
  const int k0 = n - f - 2 > 0 ? n - f - 2 : 0;
  double s = 0.0;
  int kth = k0 - 1;  // position in row i's ranking of its k-th nearest remaining
  if (i < n)
    for (int r = 0; r < k0; ++r) s += D[i * n + order[i * n + r]];
  uint64_t active = n == 64 ? ~uint64_t{0} : (uint64_t{1} << n) - 1;
  uint64_t picked = 0;
  int p = 0;
  for (int round = 0; round < rounds; ++round) {
    const bool mine = i < n && ((active >> i) & 1);
    if (round > 0 && mine) {
      const int k = n - round - f - 2;  // neighbours this round (one fewer than last round)
      if (k <= 0) {
        s = 0.0;
      } else if (pos[i * n + p] < kth) {
        s -= D[i * n + p];
      } else {
        s -= D[i * n + order[i * n + kth]];
        do {
          --kth;
        } while (kth >= 0 && !((active >> order[i * n + kth]) & 1));
      }
      // One neighbour: the score is that one distance, exactly (the subtractions
      // above leave fp64 rounding), so that two mutual nearest neighbours tie
      // exactly and the lower index decides, as in the definition.
      if (k == 1) s = D[i * n + order[i * n + kth]];
    }
    p = __builtin_amdgcn_readfirstlane(wave_argmin_lane(mine ? s : __builtin_inf()));
    if (p >= n) break;  // no vector left (rounds <= n - f keeps this from happening)
    active &= ~(uint64_t{1} << p);
    picked |= uint64_t{1} << p;
  }
  return picked;
}

__global__ __launch_bounds__(kSelectThreads) void k_bulyan_select(DistSums ds, int f, int rounds,
                                                          int32_t* __restrict__ sel) {
  const int n = ds.n;
  __shared__ double D[kNmax * kNmax];
  __shared__ unsigned char order[kNmax * kNmax];
  __shared__ unsigned char pos[kNmax * kNmax];
  load_and_rank(ds, D, order, pos);
  if (threadIdx.x >= 64) return;  // no barrier follows; wave 0 stays whole
  write_selected(krum_rounds_mask(D, order, pos, n, f, rounds), n, nullptr, sel);
}

// Contraction (many nodes, each aggregating its peers): workgroup v gathers the
// distances among its q peers (peers[v*q .. v*q+q-1], rows of the N-row input
// whose distance sums are ds) into LDS and selects among them, ties going to
// the earlier position in the peer list; sel[v*kout ..] receives the chosen
// rows as input-row indices, ascending. rounds > 0: that many rounds of
// iterated Krum; else one-shot Multi-Krum with m.
__global__ __launch_bounds__(kBlock) void k_peer_select(DistSums ds,
                                                        const int32_t* __restrict__ peers, int q,
                                                        int f, int m, int rounds, int kout,
                                                        int32_t* __restrict__ sel) {
  __shared__ double D[kNmax * kNmax];
  __shared__ unsigned char order[kNmax * kNmax];
  __shared__ unsigned char pos[kNmax * kNmax];
  __shared__ double score[kNmax];
  __shared__ int flag[kNmax];
  __shared__ int32_t map[kNmax];
  const int v = blockIdx.x;
  if (static_cast<int>(threadIdx.x) < q) {
    const int r = peers[static_cast<int64_t>(v) * q + threadIdx.x];
    map[threadIdx.x] = r < 0 ? 0 : (r >= ds.n ? ds.n - 1 : r);
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < q * q; idx += blockDim.x) {
    const int a = idx / q, b = idx % q;
    D[idx] = a == b ? 0.0 : dist_entry(ds, map[a], map[b]);
  }
  __syncthreads();
  rank_rows(D, q, order, pos);
  int32_t* out = sel + static_cast<int64_t>(v) * kout;
  if (rounds > 0) {
    if (threadIdx.x >= 64) return;
    write_selected(krum_rounds_mask(D, order, pos, q, f, rounds), q, map, out);
  } else {
    krum_flags(D, order, q, f, m, score, flag);
    if (threadIdx.x >= 64) return;
    const uint64_t mask = __ballot(static_cast<int>(threadIdx.x) < q && flag[threadIdx.x]);
    write_selected(mask, q, map, out);
  }
}

// ---------------------------------------------------------------------------
// MDA. Subsets of size s = n-f are ranked in lexicographic order; thread g
// scans ranks [g*per, (g+1)*per) with a successor step, keeping the first
// strictly smaller diameter; blocks then take the minimum (diameter, rank).

// C(a, b) for 0 <= b <= a <= kNmax (C(64, 32) < 2^61), Pascal's triangle
// built at compile time and read from constant memory: unranking takes no
// 64-bit divisions.
struct BinomTable {
  int64_t c[kNmax + 1][kNmax + 1];
};
constexpr BinomTable make_binom_table() {
  BinomTable t{};
  for (int a = 0; a <= kNmax; ++a) {
    t.c[a][0] = 1;
    for (int b = 1; b <= a; ++b) t.c[a][b] = t.c[a - 1][b - 1] + (b < a ? t.c[a - 1][b] : 0);
  }
  return t;
}
__constant__ BinomTable kBinom = make_binom_table();

__device__ __forceinline__ int64_t binom_dev(int a, int b) {
  return (b < 0 || b > a) ? 0 : kBinom.c[a][b];
}

// A thread's per-position values in LDS, position a at a stride of kBlock
// elements (neighbouring threads read neighbouring elements: no bank
// conflicts).
template <typename T>
struct Strided {
  T* base;
  __device__ T& operator[](int a) const { return base[a * kBlock]; }
};
using StridedIdx = Strided<unsigned char>;

// The rank-th s-subset of {0..n-1} in lexicographic order (rank < C(n, s)).
// Every loop is bounded by n, so an out-of-range rank cannot hang a thread;
// it yields the last subset instead.
template <typename Idx>
__device__ void unrank_subset(int64_t rank, int n, int s, Idx idx) {
  int e = 0;
  for (int t = 0; t < s; ++t) {
    const int last = n - s + t;  // largest element position t can hold
    while (e < last) {
      const int64_t cnt = binom_dev(n - e - 1, s - t - 1);
      if (rank < cnt) break;
      rank -= cnt;
      ++e;
    }
    idx[t] = static_cast<unsigned char>(e);
    ++e;
  }
}

// Lexicographic rank of positions u+1 .. s-1 of idx among the (s-1-u)-subsets
// of {idx[u]+1, ..., n-1}.
__device__ int64_t suffix_rank(int n, int s, StridedIdx idx, int u) {
  int64_t q = 0;
  for (int w = u + 1; w < s; ++w)
    for (int e = idx[w - 1] + 1; e < idx[w]; ++e) q += binom_dev(n - 1 - e, s - 1 - w);
  return q;
}

// The bound shared by a workgroup's scans: the bits of a non-negative double,
// which order as the doubles do; none (+inf) when bound is null.
__device__ __forceinline__ double read_bound(const unsigned long long* bound) {
  if (!bound) return __builtin_inf();
  const unsigned long long bits = *static_cast<const volatile unsigned long long*>(bound);
  return __longlong_as_double(static_cast<long long>(bits));
}
__device__ __forceinline__ void lower_bound_to(unsigned long long* bound, double v) {
  if (bound) atomicMin(bound, static_cast<unsigned long long>(__double_as_longlong(v)));
}

// Scan ranks [r0, r1) of the s-subsets of {0..n-1} (D: n x n in LDS, zero
// diagonal), keeping the first strictly smaller diameter: *best, *best_r
// (unchanged if r0 >= r1). Branch and bound over the lexicographic order:
// pm[u] is the D entry (row * n + column) of the largest distance among
// positions 0..u (entry 0, the zero diagonal, while there is no pair), and a
// successor step that changed position t recomputes levels t.. with one
// column of distances each. No subset extending a prefix 0..u can be the
// winner once the prefix reaches this thread's best so far (found at a lower
// rank) or exceeds *bound, the diameter of some subset (the workgroup's
// seed and every best its threads have found). Those subsets have consecutive
// ranks, the current one and the C(n-1-idx[u], s-1-u) - 1 - q after it (q,
// the rank of the current suffix among them, is 0 after a successor step),
// and the scan jumps past them. The result is the exhaustive scan's.
__device__ void mda_scan(const double* D, int n, int s, int64_t r0, int64_t r1, StridedIdx idx,
                         Strided<uint16_t> pm, unsigned long long* bound, double* best,
                         int64_t* best_r) {
  if (r0 >= r1) return;
  unrank_subset(r0, n, s, idx);
  int64_t r = r0;
  int t = 0;  // first position whose prefix maximum is stale
  bool first = true;
  for (;;) {
    const double B = read_bound(bound);
    int e = t > 0 ? pm[t - 1] : 0;
    double v = D[e];
    int u = t;
    for (; u < s; ++u) {
      const int iu = idx[u];
      const double* row = D + iu * n;
      for (int a = 0; a < u; ++a) {
        const int ia = idx[a];
        const double w = row[ia];
        if (w > v) {
          v = w;
          e = iu * n + ia;
        }
      }
      pm[u] = static_cast<uint16_t>(e);
      if (v > B || v >= *best) break;
    }
    if (u < s) {  // no subset with the prefix 0..u wins: jump to its last one
      const int64_t q = first ? suffix_rank(n, s, idx, u) : 0;
      r += binom_dev(n - 1 - idx[u], s - 1 - u) - 1 - q;
      for (int w = u + 1; w < s; ++w) idx[w] = static_cast<unsigned char>(n - s + w);
    } else if (v < *best) {
      *best = v;
      *best_r = r;
      lower_bound_to(bound, v);
    }
    first = false;
    if (r + 1 >= r1) break;
    // lexicographic successor
    t = s - 1;
    while (t >= 0 && idx[t] == n - s + t) --t;
    if (t < 0) break;
    idx[t] = static_cast<unsigned char>(idx[t] + 1);
    for (int w = t + 1; w < s; ++w) idx[w] = static_cast<unsigned char>(idx[w - 1] + 1);
    ++r;
  }
}

// Sets *bound (LDS) to an upper bound on the least diameter, before the scans
// (all threads take part; ends with a barrier). With seed, every point i is a
// center: the diameter of its s nearest points (its D row ranked, ties to the
// lower index) is the diameter of a subset, and the bound is the least of
// them. A wave takes one center at a time: lane j ranks point j (every lane
// reads the same row entry), the members form a ballot, and lane a takes the
// largest distance from member a to the members (down the columns of the
// symmetric D: consecutive lanes, consecutive banks). Without seed the bound
// starts at +inf.
__device__ void init_bound(const double* D, int n, int s, bool seed, unsigned long long* bound) {
  if (threadIdx.x == 0)
    *bound = static_cast<unsigned long long>(__double_as_longlong(__builtin_inf()));
  __syncthreads();
  if (seed) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6, waves = blockDim.x >> 6;
    double least = __builtin_inf();
    for (int i = wave; i < n; i += waves) {  // wave-uniform
      const double* row = D + i * n;
      bool in = false;
      if (lane < n) {
        const double dj = row[lane];
        int c = 0;
        for (int k = 0; k < n; ++k) {
          const double dk = row[k];
          c += (dk < dj || (dk == dj && k < lane)) ? 1 : 0;
        }
        in = c < s;
      }
      const uint64_t mem = __ballot(in);
      double v = 0.0;
      if (in)
        for (int b = 0; b < n; ++b) {
          const double w = ((mem >> b) & 1) ? D[b * n + lane] : 0.0;
          v = w > v ? w : v;
        }
#pragma unroll
      for (int m = 32; m > 0; m >>= 1) {
        const double o = __shfl_xor(v, m, 64);
        v = o > v ? o : v;
      }
      least = v < least ? v : least;
    }
    if (lane == 0 && least < __builtin_inf()) lower_bound_to(bound, least);
  }
  __syncthreads();
}

// Dynamic LDS of the subset searches: D (n x n fp64), then every thread's
// prefix maxima (s x kBlock uint16) and indices (s x kBlock bytes).
size_t scan_lds_bytes(int n, int s) {
  return static_cast<size_t>(n) * n * sizeof(double) +
         static_cast<size_t>(s) * kBlock * (sizeof(uint16_t) + 1);
}
struct ScanLds {
  double* D;
  Strided<uint16_t> pm;
  StridedIdx idx;
};
__device__ __forceinline__ ScanLds carve_scan_lds(double* lds, int n, int s) {
  uint16_t* pm = reinterpret_cast<uint16_t*>(lds + n * n);
  unsigned char* idx = reinterpret_cast<unsigned char*>(pm + s * kBlock);
  return ScanLds{lds, Strided<uint16_t>{pm + threadIdx.x}, StridedIdx{idx + threadIdx.x}};
}

// Minimum (diameter, rank) over the kBlock threads' candidates by a tree (the
// minimum of such pairs does not depend on the order of the comparisons);
// every thread receives it.
__device__ void block_min_pair(double* rd, int64_t* rr, double* best, int64_t* best_r) {
  rd[threadIdx.x] = *best;
  rr[threadIdx.x] = *best_r;
  __syncthreads();
  for (int h = kBlock / 2; h > 0; h >>= 1) {
    if (static_cast<int>(threadIdx.x) < h) {
      const int o = threadIdx.x + h;
      if (rd[o] < rd[threadIdx.x] || (rd[o] == rd[threadIdx.x] && rr[o] < rr[threadIdx.x])) {
        rd[threadIdx.x] = rd[o];
        rr[threadIdx.x] = rr[o];
      }
    }
    __syncthreads();
  }
  *best = rd[0];
  *best_r = rr[0];
}

// With one workgroup (sel non-null) it also writes the winner: the pick
// kernel is not needed.
__global__ __launch_bounds__(kBlock) void k_mda_search(DistSums ds, int s, int64_t total,
                                                       int64_t per, double* __restrict__ bdiam,
                                                       int64_t* __restrict__ brank,
                                                       int32_t* __restrict__ sel) {
  extern __shared__ double lds[];
  __shared__ double rd[kBlock];
  __shared__ int64_t rr[kBlock];
  const int n = ds.n;
  const ScanLds sl = carve_scan_lds(lds, n, s);
  load_dist(ds, sl.D);
  const int64_t g = static_cast<int64_t>(blockIdx.x) * kBlock + threadIdx.x;
  const int64_t r0 = g * per;
  const int64_t r1 = (r0 + per < total) ? r0 + per : total;
  // one subset per thread: nothing to prune, no shared bound
  __shared__ unsigned long long bound;
  unsigned long long* bp = per > 1 ? &bound : nullptr;
  if (bp) init_bound(sl.D, n, s, true, bp);
  double best = __builtin_inf();
  int64_t best_r = INT64_MAX;
  mda_scan(sl.D, n, s, r0, r1, sl.idx, sl.pm, bp, &best, &best_r);
  block_min_pair(rd, rr, &best, &best_r);
  if (sel) {
    __shared__ unsigned char win[kNmax];
    if (threadIdx.x == 0) unrank_subset(best_r, n, s, win);
    __syncthreads();
    if (static_cast<int>(threadIdx.x) < s) sel[threadIdx.x] = win[threadIdx.x];
    return;
  }
  if (threadIdx.x == 0) {
    bdiam[blockIdx.x] = best;
    brank[blockIdx.x] = best_r;
  }
}

constexpr int64_t kPeerBoundMinPer = 4;

// Contraction with MDA: workgroup v searches the C(q, f) subsets of its q
// peers (positions in the peer list, distances gathered as k_peer_select
// gathers them) for the least diameter, ties to the lowest lexicographic rank
// of positions, and writes the s = q - f chosen rows to sel[v*s ..] as
// input-row indices, ascending.
__global__ __launch_bounds__(kBlock) void k_peer_mda(DistSums ds, const int32_t* __restrict__ peers,
                                                     int q, int f, int64_t total,
                                                     int32_t* __restrict__ sel) {
  extern __shared__ double lds[];
  __shared__ double rd[kBlock];
  __shared__ int64_t rr[kBlock];
  __shared__ int32_t map[kNmax];
  const int v = blockIdx.x, s = q - f;
  const ScanLds sl = carve_scan_lds(lds, q, s);
  double* D = sl.D;
  if (static_cast<int>(threadIdx.x) < q) {
    const int r = peers[static_cast<int64_t>(v) * q + threadIdx.x];
    map[threadIdx.x] = r < 0 ? 0 : (r >= ds.n ? ds.n - 1 : r);
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < q * q; idx += blockDim.x) {
    const int a = idx / q, b = idx % q;
    D[idx] = a == b ? 0.0 : dist_entry(ds, map[a], map[b]);
  }
  __syncthreads();
  const int64_t per = (total + kBlock - 1) / kBlock;
  const int64_t r0 = static_cast<int64_t>(threadIdx.x) * per;
  const int64_t r1 = (r0 + per < total) ? r0 + per : total;
  // one workgroup per node: with a few subsets per thread the seed and the
  // shared bound cost more than they prune
  __shared__ unsigned long long bound;
  unsigned long long* bp = per > kPeerBoundMinPer ? &bound : nullptr;
  if (bp) init_bound(D, q, s, true, bp);
  double best = __builtin_inf();
  int64_t best_r = INT64_MAX;
  mda_scan(D, q, s, r0, r1, sl.idx, sl.pm, bp, &best, &best_r);
  block_min_pair(rd, rr, &best, &best_r);
  __shared__ unsigned char win[kNmax];
  if (threadIdx.x == 0) unrank_subset(best_r, q, s, win);
  __syncthreads();
  if (threadIdx.x >= 64) return;  // no barrier follows; wave 0 stays whole
  uint64_t mask = 0;
  for (int t = 0; t < s; ++t) mask |= uint64_t{1} << win[t];
  write_selected(mask, q, map, sel + static_cast<int64_t>(v) * s);
}

// At most this many search workgroups. Short ranges per thread spread over
// many workgroups beat long ones: the lanes of a wave take different successor
// steps, so a wave pays for its slowest lane at every step. Of 256 to 65536,
// 4096 was fastest from 2.6 to 621 million subsets.
constexpr int64_t kMdaMaxBlocks = 4096;

// The minimum (diameter, rank) over the search's per-workgroup results: each
// thread takes every kBlock-th workgroup, eight loads in flight at a time,
// then the block's tree; thread 0 unranks the winner.
__global__ __launch_bounds__(kBlock) void k_mda_pick(const double* __restrict__ bdiam,
                                                     const int64_t* __restrict__ brank,
                                                     int blocks, int n, int s,
                                                     int32_t* __restrict__ sel) {
  __shared__ double rd[kBlock];
  __shared__ int64_t rr[kBlock];
  __shared__ unsigned char idx[kNmax];
  constexpr int kInFlight = 8;
  double best = __builtin_inf();
  int64_t best_r = INT64_MAX;
  for (int b0 = threadIdx.x; b0 < blocks; b0 += kInFlight * kBlock) {
    double bd[kInFlight];
    int64_t br[kInFlight];
#pragma unroll
    for (int u = 0; u < kInFlight; ++u) {
      const int b = b0 + u * kBlock;
      bd[u] = b < blocks ? bdiam[b] : __builtin_inf();
      br[u] = b < blocks ? brank[b] : INT64_MAX;
    }
#pragma unroll
    for (int u = 0; u < kInFlight; ++u)
      if (bd[u] < best || (bd[u] == best && br[u] < best_r)) {
        best = bd[u];
        best_r = br[u];
      }
  }
  block_min_pair(rd, rr, &best, &best_r);
  if (threadIdx.x == 0) unrank_subset(best_r, n, s, idx);
  __syncthreads();
  if (static_cast<int>(threadIdx.x) < s) sel[threadIdx.x] = idx[threadIdx.x];
}

// ---------------------------------------------------------------------------
// MDA without enumerating the subsets, for large C(n, f). A subset S of s =
// n - f vectors has diameter at most delta exactly when the f vectors outside
// it touch every pair farther apart than delta: they form a vertex cover of
// the graph of those pairs. So the least diameter delta* is the smallest pair
// distance (or 0) whose "farther than" graph has a vertex cover of at most f
// vertices -- a binary search over the distances sorted in descending order
// -- and the winner, the lexicographically first subset of diameter delta*,
// is built vertex by vertex: v joins S (its far neighbours leave it) whenever
// the vertices still undecided can then be covered within what is left of the
// budget, else v leaves. Including the smallest possible vertex at every step
// gives the lexicographically first subset, and every step keeps a completion
// of exactly s vertices available, so the result is the enumeration's.
constexpr int kCoverThreads = 1024;

__device__ __forceinline__ uint64_t low_bits(int n) {
  return n >= 64 ? ~uint64_t{0} : (uint64_t{1} << n) - 1;
}

// One root-to-leaf path of the bounded search tree for a cover of at most k
// more vertices than c: at step t the first uncovered pair (u, v) (u the
// lowest vertex with an uncovered pair, v its lowest such neighbour) puts v
// in the cover if bit t of `path` is set, else u. True if the path covers
// every pair.
__device__ bool cover_path(const uint64_t* adj, uint64_t U, uint64_t c, int k, int64_t path) {
  for (int step = 0;; ++step) {
    int u = -1;
    uint64_t nb = 0;
    for (uint64_t cand = U & ~c; cand; cand &= cand - 1) {
      const int w = __builtin_ctzll(cand);
      const uint64_t e = adj[w] & ~c;
      if (e) {
        u = w;
        nb = e;
        break;
      }
    }
    if (u < 0) return true;
    if (step >= k) return false;
    const int v = __builtin_ctzll(nb);
    c |= ((path >> step) & 1) ? (uint64_t{1} << v) : (uint64_t{1} << u);
  }
}

// Whether at most f - |F| of the vertices outside S and F cover every pair
// among them farther apart than delta (the pairs reaching S or F are settled
// by the caller). All threads of the workgroup call it with the same
// arguments and get the same answer. First the vertices with more uncovered
// pairs than the budget go into the cover, all of them at once and again
// until none is left (any cover within the budget contains each of them):
// every wave does this alone, lane u holding vertex u's neighbours, so the
// waves agree without a barrier. Then, unless no pair is left or more pairs
// are left than the budget's vertices can touch, the 2^k paths of the search
// tree are spread over the threads, a round of them at a time, until one
// covers everything.
__device__ bool cover_feasible(const double* D, int n, double delta, uint64_t S, uint64_t F, int f,
                               uint64_t* adj) {
  const uint64_t U = low_bits(n) & ~S & ~F;
  int k = f - __popcll(F);
  if (k < 0 || k > 40) return false;  // f <= 16 under the subset limit of the entry points
  const int t = threadIdx.x, lane = t & 63;
  const bool live = lane < n && ((U >> lane) & 1);
  uint64_t a = 0;
  if (live) {
    const double* row = D + lane * n;
    for (int v = 0; v < n; ++v)
      a |= static_cast<uint64_t>(v != lane && ((U >> v) & 1) && row[v] > delta) << v;
  }
  if (t < 64) adj[t] = a;
  uint64_t C = 0;
  for (;;) {
    const uint64_t forced = __ballot(live && __popcll(a & ~C) > k && !((C >> lane) & 1));
    if (!forced) break;
    C |= forced;
    k -= __popcll(forced);
    if (k < 0) break;
  }
  bool found = false;
  if (k >= 0) {
    const bool rest = live && !((C >> lane) & 1);
    const int deg = rest ? __popcll(a & ~C) : 0;
    int edges = deg, dmax = deg;
#pragma unroll
    for (int m = 32; m > 0; m >>= 1) {
      edges += __shfl_xor(edges, m, 64);
      const int o = __shfl_xor(dmax, m, 64);
      dmax = o > dmax ? o : dmax;
    }
    edges /= 2;
    if (edges == 0) {
      found = true;
    } else if (edges <= k * dmax) {
      __syncthreads();  // adj written
      const int64_t paths = int64_t{1} << k;
      const int64_t rounds = (paths + kCoverThreads - 1) / kCoverThreads;
      for (int64_t r = 0; r < rounds; ++r) {
        const int64_t path = r * kCoverThreads + t;
        const bool mine = path < paths && cover_path(adj, U, C, k, path);
        if (__syncthreads_or(mine)) {
          found = true;
          break;
        }
      }
    }
  }
  __syncthreads();  // adj is rebuilt by the next call
  return found;
}

__global__ __launch_bounds__(kCoverThreads) void k_mda_cover(DistSums ds, int f,
                                                             int32_t* __restrict__ sel) {
  __shared__ double D[kNmax * kNmax];
  __shared__ double dv[kNmax * (kNmax - 1) / 2 + 1];
  __shared__ uint64_t adj[kNmax];
  const int n = ds.n, s = n - f, P = n * (n - 1) / 2;
  load_dist(ds, D);
  // the pair distances in descending order (equal ones by pair index), then 0
  for (int p = threadIdx.x; p < P; p += blockDim.x) {
    int i = 0, rem = p;
    while (rem >= n - 1 - i) {
      rem -= n - 1 - i;
      ++i;
    }
    const double v = D[i * n + i + 1 + rem];
    int rank = 0, q = 0;
    for (int a = 0; a < n; ++a)
      for (int b = a + 1; b < n; ++b, ++q) {
        const double w = D[a * n + b];
        rank += (w > v) | ((w == v) & (q < p));
      }
    dv[rank] = v;
  }
  if (threadIdx.x == 0) dv[P] = 0.0;
  __syncthreads();
  // largest j whose distance dv[j] admits a cover (j = 0 always does: no pair
  // is farther apart than the largest distance)
  int lo = 0, hi = P;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (cover_feasible(D, n, dv[mid], 0, 0, f, adj)) lo = mid;
    else hi = mid - 1;
  }
  const double delta = dv[lo];
  uint64_t S = 0, F = 0;
  for (int v = 0; v < n; ++v) {
    const uint64_t rest = low_bits(n) & ~S & ~F;
    if (__popcll(S) == s) {
      F |= rest;
      break;
    }
    if (__popcll(F) == f) {
      S |= rest;
      break;
    }
    const int lane = threadIdx.x & 63;  // every wave forms the same mask
    const uint64_t far = __ballot(lane < n && lane != v && D[v * n + lane] > delta);
    const uint64_t bit = uint64_t{1} << v;
    if (far & S) {
      F |= bit;
      continue;
    }
    const uint64_t S2 = S | bit, F2 = F | (far & rest & ~bit);
    if (__popcll(F2) <= f && cover_feasible(D, n, delta, S2, F2, f, adj)) {
      S = S2;
      F = F2;
    } else {
      F |= bit;
    }
  }
  // S has exactly s members; the clamp only guards the sel writes
  while (__popcll(S) > s) S &= ~(uint64_t{1} << (63 - __builtin_clzll(S)));
  if (threadIdx.x < 64) write_selected(S, n, nullptr, sel);
}

// Dynamic LDS above 64 KB (n near 64 with large s) is requested from the
// runtime first.
hipError_t allow_lds(const void* kernel, size_t bytes) {
  if (bytes <= 65536) return hipSuccess;
  return hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                             static_cast<int>(bytes));
}

void mda_split(int n, int f, int64_t* total, int64_t* per, int* blocks) {
  *total = binomial(n, f);
  *per = (*total + kMdaMaxBlocks * kBlock - 1) / (kMdaMaxBlocks * kBlock);
  if (*per < 1) *per = 1;
  *blocks = static_cast<int>((*total + *per * kBlock - 1) / (*per * kBlock));
}

}  // namespace

int64_t binomial(int a, int b) {
  if (b < 0 || b > a) return 0;
  if (b > a - b) b = a - b;
  unsigned __int128 c = 1;
  for (int t = 1; t <= b; ++t) {
    c = c * static_cast<unsigned>(a - b + t) / static_cast<unsigned>(t);
    if (c > (static_cast<unsigned __int128>(1) << 62)) return -1;
  }
  return static_cast<int64_t>(c);
}

int mda_blocks(int n, int f) {
  int64_t total, per;
  int blocks;
  mda_split(n, f, &total, &per, &blocks);
  return blocks;
}

size_t mda_scratch_bytes(int n, int f) {
  if (mda_uses_cover(n, f)) return 0;
  return static_cast<size_t>(mda_blocks(n, f)) * (sizeof(double) + sizeof(int64_t));
}

hipError_t enqueue_krum_select(const DistSums& ds, int f, int m, int32_t* sel, hipStream_t s) {
  launch("krum_select", k_krum_select, dim3(1), dim3(kSelectThreads), 0, s, ds, f, m, sel);
  return hipGetLastError();
}

namespace {
bool g_fused = true;
}  // namespace

bool fused_enabled() { return __atomic_load_n(&g_fused, __ATOMIC_RELAXED); }
void set_fused(bool on) { __atomic_store_n(&g_fused, on, __ATOMIC_RELAXED); }

bool krum_fusable(const DistPlan& p, const float* out) {
  if (!fused_enabled() || p.engine != kEngineDirect || p.n < 3 || p.n > kFusedMaxN ||
      p.width != 4 || p.tiles > kFoldTiles || !out || load_width(out) != 4)
    return false;
  // every workgroup reads all tile partials: keep that repeated read small
  const double reread = static_cast<double>(select_mean_groups(p.d)) * p.entries * p.tiles * 8.0;
  return reread <= kFusedRereadBytes;
}

hipError_t enqueue_krum_select_mean(const float* x, const DistSums& ds, int64_t d, int f, int m,
                                    int32_t* sel, float* out, hipStream_t s) {
  if (!ds.partial || ds.engine != kEngineDirect || !sel || !out) return hipErrorInvalidValue;
  return select_mean_dispatch<3>(ds.n, x, d, ds, f, m, sel, out, s);
}

hipError_t enqueue_bulyan_select(const DistSums& ds, int f, int32_t* sel, hipStream_t s) {
  launch("bulyan_select", k_bulyan_select, dim3(1), dim3(kSelectThreads), 0, s, ds, f,
         ds.n - 2 * f, sel);
  return hipGetLastError();
}

hipError_t enqueue_krum_rounds(const DistSums& ds, int f, int rounds, int32_t* sel,
                               hipStream_t s) {
  launch("krum_rounds", k_bulyan_select, dim3(1), dim3(kSelectThreads), 0, s, ds, f, rounds, sel);
  return hipGetLastError();
}

hipError_t enqueue_peer_select(const DistSums& ds, int nodes, const int32_t* peers, int q, int f,
                               int m, int rounds, int kout, int32_t* sel, hipStream_t s) {
  launch("peer_select", k_peer_select, dim3(nodes), dim3(kBlock), 0, s, ds, peers, q, f, m, rounds,
         kout, sel);
  return hipGetLastError();
}

hipError_t enqueue_peer_mda(const DistSums& ds, int nodes, const int32_t* peers, int q, int f,
                            int32_t* sel, hipStream_t s) {
  const int64_t total = binomial(q, f);
  if (total < 1) return hipErrorInvalidValue;
  const size_t lds = scan_lds_bytes(q, q - f);
  hipError_t e = allow_lds(reinterpret_cast<const void*>(k_peer_mda), lds);
  if (e != hipSuccess) return e;
  launch("peer_mda", k_peer_mda, dim3(nodes), dim3(kBlock), static_cast<uint32_t>(lds), s, ds,
         peers, q, f, total, sel);
  return hipGetLastError();
}

namespace {
int64_t g_mda_cover_min = int64_t{1} << 20;
}  // namespace

int64_t mda_cover_min() { return __atomic_load_n(&g_mda_cover_min, __ATOMIC_RELAXED); }
void set_mda_cover_min(int64_t subsets) {
  __atomic_store_n(&g_mda_cover_min, subsets, __ATOMIC_RELAXED);
}

bool mda_uses_cover(int n, int f) {
  const int64_t total = binomial(n, f);
  return total < 0 || total >= mda_cover_min();
}

hipError_t enqueue_mda_select(const DistSums& ds, int f, void* scratch, int32_t* sel,
                              hipStream_t s) {
  const int n = ds.n;
  if (mda_uses_cover(n, f)) {
    launch("mda_cover", k_mda_cover, dim3(1), dim3(kCoverThreads), 0, s, ds, f, sel);
    return hipGetLastError();
  }
  int64_t total, per;
  int blocks;
  mda_split(n, f, &total, &per, &blocks);
  double* bdiam = static_cast<double*>(scratch);
  int64_t* brank = reinterpret_cast<int64_t*>(bdiam + blocks);
  const size_t lds = scan_lds_bytes(n, n - f);
  hipError_t e = allow_lds(reinterpret_cast<const void*>(k_mda_search), lds);
  if (e != hipSuccess) return e;
  launch("mda_search", k_mda_search, dim3(blocks), dim3(kBlock), static_cast<uint32_t>(lds), s, ds,
         n - f, total, per, bdiam, brank, blocks == 1 ? sel : nullptr);
  e = hipGetLastError();
  if (e != hipSuccess || blocks == 1) return e;
  launch("mda_pick", k_mda_pick, dim3(1), dim3(kBlock), 0, s, bdiam, brank, blocks, n, n - f, sel);
  return hipGetLastError();
}

}  // namespace garfield
