// Plain CPU oracle for the Garfield gradient aggregation rules (GARs).
//
// TEST INFRASTRUCTURE ONLY. Nothing on the product path may link, load or call
// this file; only the test suite, the smoke check and the benchmark's CPU
// baseline leg use it. It shares no code with the HIP library.
//
// Conventions (one rule for every function below):
//   * inputs are n x d fp32 vectors, row-major (row i starts at x + i*d);
//   * every value is widened exactly to fp64 and all arithmetic is fp64;
//   * aggregates are rounded once, to nearest-even fp32, at the very end;
//   * index outputs are sets, written in ascending order;
//   * the only parallelism is the one the paper gives for its CPU median
//     (each core takes a contiguous share of coordinates, Section 4.3), and a
//     parallel loop over independent vector pairs for the distances. Neither
//     changes the order of any floating-point sum.
//
// Readings of the paper used where it is silent (each is listed in the design
// notes of the repository):
//   R1  Krum's distance is the squared Euclidean distance.
//   R2  Krum's score sums the n-f-2 smallest distances to the *other* vectors,
//       added in ascending order.
//   R3  ties in a score ordering are broken towards the lower index.
//   R4  Multi-Krum is one-shot: the m lowest (score, index) pairs; m defaults
//       to n-f.
//   R5  the median of an even count is the mean of the two middle values.
//   R6  Bulyan: theta = n-2f rounds of Krum on the not-yet-selected set with
//       n_R-f-2 neighbours (clamped at 0), then per coordinate the
//       beta = theta-2f values closest to the median under the key
//       (|v - med|, v), averaged.
//   R8  iterated Multi-Krum: the selection of R6 stopped after m rounds, then
//       the mean of the m selected rows (Multi-Krum computed by repeating
//       Krum, as Section 4.4 describes for Multi-Krum and Bulyan).
//   R9  attacks (Section 3.2, Main objects; Section 6.5): reversed vectors are
//       param times an honest vector (row b uses honest row b mod h); random
//       vectors are param times standard normals drawn by Box-Muller from
//       Philox4x32-10 words (counter = (c/4 low, c/4 high, b, 0), key = seed;
//       a word w becomes the uniform ((w >> 9) + 1/2) 2^-23); "little is
//       enough" is mean - param * std per coordinate with the population
//       standard deviation; "fall of empires" is -param * mean.
//   R10 variance condition (Section 3.1, Tradeoffs): sigma^2 = E||g - E g||^2
//       is estimated without bias over the h honest vectors,
//       sum_i ||g_i - mean||^2 / (h - 1).
//   R7  MDA enumerates the subsets of size n-f in lexicographic order and keeps
//       the first one of strictly smaller diameter (diameter = largest squared
//       distance inside the subset).
//
// Status codes match the library's: 0 ok, 1 invalid argument, 2 n too small
// for the rule's requirement in f.

#include <omp.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <utility>
#include <vector>

namespace {

constexpr int kOk = 0;
constexpr int kInval = 1;
constexpr int kReq = 2;

inline double at(const float* x, int64_t d, int i, int64_t c) {
  return static_cast<double>(x[static_cast<int64_t>(i) * d + c]);
}

// Squared Euclidean distance between rows i and j, summed over c = 0..d-1 in
// order (Section 3.1, items 2-4 use this distance).
double sqdist(const float* x, int64_t d, int i, int j) {
  double s = 0.0;
  for (int64_t c = 0; c < d; ++c) {
    const double t = at(x, d, i, c) - at(x, d, j, c);
    s += t * t;
  }
  return s;
}

// Full symmetric distance matrix with a zero diagonal.
void distance_matrix(const float* x, int n, int64_t d, double* D) {
  std::vector<std::pair<int, int>> pairs;
  for (int i = 0; i < n; ++i)
    for (int j = i + 1; j < n; ++j) pairs.emplace_back(i, j);
  for (int i = 0; i < n; ++i) D[i * n + i] = 0.0;
  const int64_t np = static_cast<int64_t>(pairs.size());
#pragma omp parallel for schedule(dynamic, 1)
  for (int64_t p = 0; p < np; ++p) {
    const int i = pairs[p].first, j = pairs[p].second;
    const double s = sqdist(x, d, i, j);
    D[i * n + j] = s;
    D[j * n + i] = s;
  }
}

// Krum score of row i against the candidate set `cand` (which contains i):
// the sum of the k smallest distances from i to the other candidates, added
// in ascending order (Section 3.1 item 2, readings R1-R2).
double krum_score(const double* D, int n, const std::vector<int>& cand, int i, int k) {
  std::vector<double> dist;
  for (int j : cand)
    if (j != i) dist.push_back(D[i * n + j]);
  std::sort(dist.begin(), dist.end());
  double s = 0.0;
  for (int t = 0; t < k && t < static_cast<int>(dist.size()); ++t) s += dist[t];
  return s;
}

// Mean of the rows in `rows` (ascending), per coordinate, rounded once.
void mean_rows(const float* x, int64_t d, const std::vector<int>& rows, float* out) {
  const double count = static_cast<double>(rows.size());
#pragma omp parallel for schedule(static)
  for (int64_t c = 0; c < d; ++c) {
    double s = 0.0;
    for (int i : rows) s += at(x, d, i, c);
    out[c] = static_cast<float>(s / count);
  }
}

// `rounds` rounds of Krum over the not-yet-selected rows (readings R6, R8):
// round r scores every remaining row against the other remaining rows with
// max(|remaining| - f - 2, 0) neighbours and moves the lowest (score, index)
// to the selection. Returns the picks in the order they were made; fills
// `picks` (rounds entries) and `round_scores` (rounds*n, +inf for rows already
// picked) when given.
std::vector<int> iterated_krum(const double* D, int n, int f, int rounds, int32_t* picks,
                               double* round_scores) {
  std::vector<int> remaining(n);
  for (int i = 0; i < n; ++i) remaining[i] = i;
  std::vector<int> chosen;
  for (int r = 0; r < rounds; ++r) {
    const int k = std::max(static_cast<int>(remaining.size()) - f - 2, 0);
    double best = 0.0;
    int best_i = -1;
    if (round_scores)
      for (int i = 0; i < n; ++i) round_scores[static_cast<int64_t>(r) * n + i] = 1.0 / 0.0;
    for (int i : remaining) {  // ascending, so strict < keeps the lower index on ties
      const double s = krum_score(D, n, remaining, i, k);
      if (round_scores) round_scores[static_cast<int64_t>(r) * n + i] = s;
      if (best_i < 0 || s < best) {
        best = s;
        best_i = i;
      }
    }
    if (picks) picks[r] = best_i;
    chosen.push_back(best_i);
    remaining.erase(std::find(remaining.begin(), remaining.end(), best_i));
  }
  return chosen;
}

// Median of k values: middle element for odd k, mean of the two middle
// elements for even k (Section 3.1 item 1, reading R5).
double median_of(std::vector<double>& v) {
  std::sort(v.begin(), v.end());
  const size_t k = v.size();
  if (k % 2 == 1) return v[k / 2];
  return (v[k / 2 - 1] + v[k / 2]) / 2.0;
}

}  // namespace

extern "C" {

// D (n*n fp64) = pairwise squared Euclidean distances.
int oracle_pairwise_sqdist(const float* x, int n, int64_t d, double* D) {
  if (n < 1 || d < 0 || !D || (d > 0 && !x)) return kInval;
  distance_matrix(x, n, d, D);
  return kOk;
}

// Krum scores of all n rows with k = n - f - 2 neighbours.
int oracle_krum_scores(const float* x, int n, int f, int64_t d, double* scores) {
  if (n < 1 || f < 0 || d < 0 || !scores || (d > 0 && !x)) return kInval;
  if (n < 2 * f + 3) return kReq;
  std::vector<double> D(static_cast<size_t>(n) * n);
  distance_matrix(x, n, d, D.data());
  std::vector<int> all(n);
  for (int i = 0; i < n; ++i) all[i] = i;
  for (int i = 0; i < n; ++i) scores[i] = krum_score(D.data(), n, all, i, n - f - 2);
  return kOk;
}

// Multi-Krum (Section 3.1 item 2): the m rows with the lowest (score, index),
// then their mean. m <= 0 selects the default n - f. Krum is m = 1.
// `scores` (n fp64) and `D_out` (n*n fp64, the distance matrix) are optional.
int oracle_multikrum(const float* x, int n, int f, int64_t d, int m, float* out,
                     int32_t* sel, double* scores, double* D_out) {
  if (n < 1 || f < 0 || d < 0 || !sel || (d > 0 && (!x || !out))) return kInval;
  if (n < 2 * f + 3) return kReq;
  if (m <= 0) m = n - f;
  if (m > n - f) return kInval;
  std::vector<double> D(static_cast<size_t>(n) * n);
  distance_matrix(x, n, d, D.data());
  if (D_out) std::copy(D.begin(), D.end(), D_out);
  std::vector<int> all(n);
  for (int i = 0; i < n; ++i) all[i] = i;
  std::vector<std::pair<double, int>> ranked;
  for (int i = 0; i < n; ++i) {
    const double s = krum_score(D.data(), n, all, i, n - f - 2);
    if (scores) scores[i] = s;
    ranked.emplace_back(s, i);
  }
  std::sort(ranked.begin(), ranked.end());  // (score, index): ties -> lower index
  std::vector<int> chosen;
  for (int t = 0; t < m; ++t) chosen.push_back(ranked[t].second);
  std::sort(chosen.begin(), chosen.end());
  for (int t = 0; t < m; ++t) sel[t] = chosen[t];
  mean_rows(x, d, chosen, out);
  return kOk;
}

// Iterated Multi-Krum (reading R8): m rounds of Krum over the rows not yet
// selected, then the mean of the m selected rows. m <= 0 selects n - f.
// `picks` (optional, m entries) receives the rows in the order they were
// picked, `round_scores` (optional, m*n fp64) every row's score per round
// (+inf for rows already picked), `D_out` (optional, n*n) the distances.
int oracle_multikrum_iterated(const float* x, int n, int f, int64_t d, int m, float* out,
                              int32_t* sel, int32_t* picks, double* round_scores,
                              double* D_out) {
  if (n < 1 || f < 0 || d < 0 || !sel || (d > 0 && (!x || !out))) return kInval;
  if (n < 2 * f + 3) return kReq;
  if (m <= 0) m = n - f;
  if (m > n - f) return kInval;
  std::vector<double> D(static_cast<size_t>(n) * n);
  distance_matrix(x, n, d, D.data());
  if (D_out) std::copy(D.begin(), D.end(), D_out);
  std::vector<int> chosen = iterated_krum(D.data(), n, f, m, picks, round_scores);
  std::sort(chosen.begin(), chosen.end());
  for (int t = 0; t < m; ++t) sel[t] = chosen[t];
  mean_rows(x, d, chosen, out);
  return kOk;
}

// Coordinate-wise median (Section 3.1 item 1) over the k rows listed in
// `rows`, or over all n rows when rows is null (then k must be n).
int oracle_median(const float* x, int n, int f, int64_t d, const int32_t* rows, int k,
                  float* out) {
  if (n < 1 || f < 0 || d < 0 || (d > 0 && (!x || !out))) return kInval;
  if (n < 2 * f + 1) return kReq;
  std::vector<int> use;
  if (rows) {
    if (k < 1) return kInval;
    for (int t = 0; t < k; ++t) {
      if (rows[t] < 0 || rows[t] >= n) return kInval;
      use.push_back(rows[t]);
    }
  } else {
    if (k != n && k > 0) return kInval;
    for (int i = 0; i < n; ++i) use.push_back(i);
  }
  // Contiguous coordinate share per core, as in the paper's CPU median.
#pragma omp parallel
  {
    std::vector<double> v(use.size());
#pragma omp for schedule(static)
    for (int64_t c = 0; c < d; ++c) {
      for (size_t t = 0; t < use.size(); ++t) v[t] = at(x, d, use[t], c);
      out[c] = static_cast<float>(median_of(v));
    }
  }
  return kOk;
}

// Bulyan (Section 3.1 item 4, reading R6). `sel` receives the theta selected
// rows in ascending order; `picks` (optional, theta entries) the same rows in
// the order they were picked; `round_scores` (optional, theta*n fp64) the
// Krum score of every row in each round, +inf for rows already picked;
// `D_out` (optional, n*n fp64) the distance matrix.
int oracle_bulyan(const float* x, int n, int f, int64_t d, float* out, int32_t* sel,
                  int32_t* picks, double* round_scores, double* D_out) {
  if (n < 1 || f < 0 || d < 0 || !sel || (d > 0 && (!x || !out))) return kInval;
  if (n < 4 * f + 3) return kReq;
  const int theta = n - 2 * f;
  const int beta = theta - 2 * f;
  std::vector<double> D(static_cast<size_t>(n) * n);
  distance_matrix(x, n, d, D.data());
  if (D_out) std::copy(D.begin(), D.end(), D_out);
  std::vector<int> chosen = iterated_krum(D.data(), n, f, theta, picks, round_scores);
  std::sort(chosen.begin(), chosen.end());
  for (int t = 0; t < theta; ++t) sel[t] = chosen[t];
#pragma omp parallel
  {
    std::vector<double> v(theta);
    std::vector<std::pair<double, double>> key(theta);
#pragma omp for schedule(static)
    for (int64_t c = 0; c < d; ++c) {
      for (int t = 0; t < theta; ++t) v[t] = at(x, d, chosen[t], c);
      std::vector<double> tmp(v);
      const double med = median_of(tmp);
      for (int t = 0; t < theta; ++t) {
        const double dist = v[t] > med ? v[t] - med : med - v[t];
        key[t] = std::make_pair(dist, v[t]);
      }
      std::sort(key.begin(), key.end());
      double s = 0.0;
      for (int t = 0; t < beta; ++t) s += key[t].second;
      out[c] = static_cast<float>(s / static_cast<double>(beta));
    }
  }
  return kOk;
}

// Minimum-diameter averaging (Section 3.1 item 3, reading R7). `best_diam`
// and `second_diam` (optional) receive the smallest diameter and the smallest
// diameter strictly larger than it (+inf if none). `n_best` (optional)
// receives how many subsets reach the smallest diameter; `D_out` (optional,
// n*n fp64) the distance matrix.
int oracle_mda(const float* x, int n, int f, int64_t d, float* out, int32_t* sel,
               double* best_diam, double* second_diam, int64_t* n_best, double* D_out) {
  if (n < 1 || f < 0 || d < 0 || !sel || (d > 0 && (!x || !out))) return kInval;
  if (n < 2 * f + 1) return kReq;
  const int s = n - f;
  std::vector<double> D(static_cast<size_t>(n) * n);
  distance_matrix(x, n, d, D.data());
  if (D_out) std::copy(D.begin(), D.end(), D_out);
  // Lexicographic enumeration of s-subsets of {0..n-1}.
  std::vector<int> idx(s);
  for (int t = 0; t < s; ++t) idx[t] = t;
  std::vector<int> best_set(idx);
  double best = 1.0 / 0.0, second = 1.0 / 0.0;
  int64_t count_best = 0;
  while (true) {
    double diam = 0.0;
    for (int a = 0; a < s; ++a)
      for (int b = a + 1; b < s; ++b) diam = std::max(diam, D[idx[a] * n + idx[b]]);
    if (diam < best) {
      second = best;
      best = diam;
      best_set = idx;
      count_best = 1;
    } else if (diam == best) {
      ++count_best;
    } else if (diam < second) {
      second = diam;
    }
    int t = s - 1;
    while (t >= 0 && idx[t] == n - s + t) --t;
    if (t < 0) break;
    ++idx[t];
    for (int u = t + 1; u < s; ++u) idx[u] = idx[u - 1] + 1;
  }
  for (int t = 0; t < s; ++t) sel[t] = best_set[t];
  if (best_diam) *best_diam = best;
  if (second_diam) *second_diam = second;
  if (n_best) *n_best = count_best;
  mean_rows(x, d, best_set, out);
  return kOk;
}

// Philox4x32-10 (Salmon, Moraes, Dror and Shaw, SC'11): ten rounds; in each,
// the products M0 * c0 and M1 * c2 (32 x 32 -> 64 bits) give the new words
// (hi(M1 c2) ^ c1 ^ k0, lo(M1 c2), hi(M0 c0) ^ c3 ^ k1, lo(M0 c0)); the key
// gains (W0, W1) before every round after the first.
void oracle_philox4x32_10(const uint32_t* ctr, const uint32_t* key, uint32_t* out) {
  const uint64_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u;
  uint32_t c[4] = {ctr[0], ctr[1], ctr[2], ctr[3]};
  uint32_t k[2] = {key[0], key[1]};
  for (int r = 0; r < 10; ++r) {
    if (r > 0) {
      k[0] += 0x9E3779B9u;
      k[1] += 0xBB67AE85u;
    }
    const uint64_t a = M0 * c[0], b = M1 * c[2];
    const uint32_t next[4] = {static_cast<uint32_t>(b >> 32) ^ c[1] ^ k[0],
                              static_cast<uint32_t>(b),
                              static_cast<uint32_t>(a >> 32) ^ c[3] ^ k[1],
                              static_cast<uint32_t>(a)};
    for (int t = 0; t < 4; ++t) c[t] = next[t];
  }
  for (int t = 0; t < 4; ++t) out[t] = c[t];
}

// Byzantine vectors (reading R9). kind: 0 reversed, 1 random, 2 little is
// enough, 3 fall of empires. honest: h x d (unused for random); byz: nbyz x d.
int oracle_attack(int kind, const float* honest, int h, int64_t d, double param, uint64_t seed,
                  float* byz, int nbyz) {
  if (kind < 0 || kind > 3 || d < 0 || nbyz < 0 || (d > 0 && nbyz > 0 && !byz)) return kInval;
  if (kind != 1 && (h < 1 || (d > 0 && !honest))) return kInval;
  const double two_pi = 6.283185307179586476925286766559;
  for (int b = 0; b < nbyz; ++b) {
    float* row = byz + static_cast<int64_t>(b) * d;
    if (kind == 0) {
      for (int64_t c = 0; c < d; ++c) row[c] = static_cast<float>(param * at(honest, d, b % h, c));
    } else if (kind == 1) {
      for (int64_t q = 0; 4 * q < d; ++q) {
        const uint32_t ctr[4] = {static_cast<uint32_t>(q), static_cast<uint32_t>(q >> 32),
                                 static_cast<uint32_t>(b), 0u};
        const uint32_t key[2] = {static_cast<uint32_t>(seed), static_cast<uint32_t>(seed >> 32)};
        uint32_t w[4];
        oracle_philox4x32_10(ctr, key, w);
        double z[4];
        for (int pair = 0; pair < 2; ++pair) {
          const double u1 = (static_cast<double>(w[2 * pair] >> 9) + 0.5) / 8388608.0;
          const double u2 = (static_cast<double>(w[2 * pair + 1] >> 9) + 0.5) / 8388608.0;
          const double r = std::sqrt(-2.0 * std::log(u1));
          z[2 * pair] = r * std::cos(two_pi * u2);
          z[2 * pair + 1] = r * std::sin(two_pi * u2);
        }
        for (int e = 0; e < 4 && 4 * q + e < d; ++e) row[4 * q + e] = static_cast<float>(param * z[e]);
      }
    } else {
      for (int64_t c = 0; c < d; ++c) {
        double sum = 0.0;
        for (int i = 0; i < h; ++i) sum += at(honest, d, i, c);
        const double mean = sum / h;
        if (kind == 3) {
          row[c] = static_cast<float>(-param * mean);
        } else {
          double ss = 0.0;
          for (int i = 0; i < h; ++i) {
            const double t = at(honest, d, i, c) - mean;
            ss += t * t;
          }
          row[c] = static_cast<float>(mean - param * std::sqrt(ss / h));
        }
      }
    }
  }
  return kOk;
}

// Variance condition (reading R10): stats[0] = sum_i ||g_i - mean||^2 / (h-1)
// over the h rows of g, stats[1] = ||grad||^2.
int oracle_variance_stats(const float* g, int h, int64_t d, const float* grad, double* stats) {
  if (h < 2 || d < 0 || !stats || (d > 0 && (!g || !grad))) return kInval;
  double dev = 0.0;
  for (int64_t c = 0; c < d; ++c) {
    double sum = 0.0;
    for (int i = 0; i < h; ++i) sum += at(g, d, i, c);
    const double mean = sum / h;
    for (int i = 0; i < h; ++i) {
      const double t = at(g, d, i, c) - mean;
      dev += t * t;
    }
  }
  double norm = 0.0;
  for (int64_t c = 0; c < d; ++c) norm += static_cast<double>(grad[c]) * static_cast<double>(grad[c]);
  stats[0] = dev / (h - 1);
  stats[1] = norm;
  return kOk;
}

// Threads of the OpenMP team that the parallel loops above run with (the
// size of a default parallel region on this host), for reporting.
int oracle_omp_team_size() {
  int team = 0;
#pragma omp parallel
  {
#pragma omp single
    team = omp_get_num_threads();
  }
  return team;
}

}  // extern "C"
