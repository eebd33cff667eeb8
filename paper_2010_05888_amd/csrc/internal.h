// Internal declarations shared by the HIP translation units of libgarfield.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

namespace garfield {

constexpr int kBlock = 256;       // threads per workgroup (4 wave64s)
constexpr int kNmax = 64;         // largest n any kernel is built for
constexpr int kDirectMaxNLimit = 20;   // direct-difference kernels are built for n <= this
constexpr int kGramBlocks = 4;    // Gram engine: at most 4 blocks of 16 rows (n <= 64)
constexpr int kProbeRuns = 4;     // reference-row probe: runs of kBlock coordinates
constexpr int kDirectLaneCoords = 16;  // direct engine: coordinates per lane per tile

// Where D comes from: nothing ran (all zero), the direct or Gram engine's
// entry sums, or a full n x n fp64 matrix (segmented aggregation).
enum Engine { kEngineNone = 0, kEngineDirect = 1, kEngineGram = 2, kEngineMatrix = 3 };

// How the distance step is tiled for (n, d).
struct DistPlan {
  int engine = kEngineNone;
  int n = 0;
  int64_t d = 0;
  int width = 1;           // floats per vector load (1, 2 or 4)
  int64_t chunk = 0;       // coordinates per workgroup (tile)
  int64_t tiles = 0;       // workgroups of the distance kernel
  int entries = 0;         // partial sums each tile writes
};

// n <= direct_max_n(): distances by direct differences on VALU; else MFMA Gram.
int direct_max_n();
void set_direct_max_n(int n);

DistPlan plan_distances(int n, int64_t d, const float* x);

// Compute units of the current device (256 on MI355X; also the fallback when
// no device is available, e.g. when only planning on a host without a GPU).
int device_cus();
// Direct engine: coordinates per tile for a segment of length d read with
// `width`-float loads.
int64_t direct_chunk(int64_t d, int width);

// Device workspace of the distance step (256-byte aligned sections).
struct DistWorkspace {
  double* partial = nullptr;  // entries x tiles (entry-major)
  double* sums = nullptr;     // entries
  double* probe = nullptr;    // kProbeRuns x kNmax x kNmax (Gram engine only)
  int32_t* ref = nullptr;     // 1 (Gram engine only)
};
struct DistSums;
size_t dist_workspace_bytes(const DistPlan& p);
DistWorkspace carve_dist_workspace(const DistPlan& p, void* base);

// Gram engine only: probe and choose the reference row into ws.ref.
hipError_t enqueue_reference(const float* x, const DistPlan& p, const DistWorkspace& ws,
                             hipStream_t s);

// Enqueue the distance step; when the stream reaches its end, ws.sums holds
// one fp64 sum per entry (see dist_layout.h for how they map to D). With
// sum_tiles false only the tiles' partials are written (the folded form).
// colsum (d doubles; direct engine with n <= kColSumMaxN only): the step also
// writes every coordinate's exact column sum of the n rows, or NaN where that
// sum or a sum of some of the rows might not be exact (ColSum in
// direct_body.h).
constexpr int kColSumMaxN = 12;
hipError_t enqueue_distances(const float* x, const DistPlan& p, const DistWorkspace& ws,
                             hipStream_t s, bool sum_tiles = true, double* colsum = nullptr);
// Direct-engine plans with at most kFoldTiles tiles and max_entries entries
// may leave the tile sums to the selection kernel (DistSums' folded form):
// its waves add four entries at a time, so a workgroup of w waves folds up to
// 4w entries in one round of loads.
constexpr int64_t kFoldTiles = 256;
bool foldable(const DistPlan& p, int max_entries);
DistSums dist_sums(const DistPlan& p, const DistWorkspace& ws);
// Write D (n x n fp64, device) from the entry sums.
hipError_t enqueue_write_dist(const DistSums& ds, double* dist, hipStream_t s);

// Multi-Krum's selection and mean in one kernel (select.hip) for short
// inputs: direct-engine plans of 3 <= n <= kFusedMaxN rows with 16-byte loads
// whose distance step leaves its tile partials folded (at most kFoldTiles
// tiles), a float-aligned out, and a repeated read of the partials (every one
// of the kernel's workgroups, one per 1,024 coordinates, adds all of them) of
// at most kFusedRereadBytes. ds: the folded distance sums of x. The selection
// and the output are bit-identical to k_krum_select's and k_mean_rows'.
constexpr int kFusedMaxN = 12;
constexpr double kFusedRereadBytes = 8.0 * 1024 * 1024;
bool fused_enabled();
void set_fused(bool on);
bool krum_fusable(const DistPlan& p, const float* out);
hipError_t enqueue_krum_select_mean(const float* x, const DistSums& ds, int64_t d, int f, int m,
                                    int32_t* sel, float* out, hipStream_t s);

// Selection on D (one workgroup each).
hipError_t enqueue_krum_select(const DistSums& ds, int f, int m, int32_t* sel, hipStream_t s);
hipError_t enqueue_bulyan_select(const DistSums& ds, int f, int32_t* sel, hipStream_t s);
// `rounds` rounds of Krum over the not-yet-selected vectors (iterated Multi-Krum).
hipError_t enqueue_krum_rounds(const DistSums& ds, int f, int rounds, int32_t* sel,
                               hipStream_t s);

// Tile partials (entry-major, `tiles` per entry) -> one fp64 sum per entry.
hipError_t enqueue_sum_tiles(const double* partial, int64_t tiles, int entries, double* sums,
                             hipStream_t s);

// Segment tables (segtable.hip): K segments of n <= kDirectMaxNLimit vectors
// stored apart, ptrs[s * n + i] -> segment s of vector i (dims[s] floats, host
// array). Distances: direct-engine tile partials, entry-major with `tiles` =
// table_tiles(dims, K, n) per entry. Aggregation: one output per segment (host
// array of device pointers).
int64_t table_tiles(const int64_t* dims, int K, int n);
hipError_t enqueue_distances_table(const float* const* ptrs, int n, const int64_t* dims, int K,
                                   double* partial, int64_t tiles, hipStream_t s);
// The Gram engine over a table (n > 20): table_gram_tiles = partial columns
// (-1 if a launch would exceed 2^31 stages); probe_space holds
// table_gram_probe_bytes() of probe matrices and the reference row; the
// partials have the Gram layout of dist_layout.h.
int64_t table_gram_tiles(const int64_t* dims, int K, int n);
size_t table_gram_probe_bytes();
hipError_t enqueue_distances_table_gram(const float* const* ptrs, int n, const int64_t* dims,
                                        int K, double* partial, int64_t tiles, void* probe_space,
                                        hipStream_t s);
// Its reference row alone (into table_reference_slot(probe_space)); needs a
// nonempty segment.
hipError_t enqueue_table_reference(const float* const* ptrs, int n, const int64_t* dims, int K,
                                   void* probe_space, hipStream_t s);
int32_t* table_reference_slot(void* probe_space);
hipError_t enqueue_mean_rows_table(const float* const* ptrs, int n, const int64_t* dims,
                                   float* const* outs, int K, const int32_t* rows, int k,
                                   hipStream_t s);
// The coordinate-wise median over all n vectors of each segment.
hipError_t enqueue_median_table(const float* const* ptrs, int n, const int64_t* dims,
                                float* const* outs, int K, hipStream_t s);
hipError_t enqueue_bulyan_table(const float* const* ptrs, int n, int f, const int64_t* dims,
                                float* const* outs, int K, const int32_t* sel, hipStream_t s);

// Contraction steps (contract.hip, k_peer_select in select.hip): `nodes`
// nodes, node v aggregating q peers (peers[v*q ..], rows of the n-row x).
// Selection: sel[v*kout ..] = node v's chosen rows, ascending; rounds > 0 is
// iterated Krum, else one-shot Multi-Krum with m. Aggregation: row v of y.
hipError_t enqueue_peer_select(const DistSums& ds, int nodes, const int32_t* peers, int q, int f,
                               int m, int rounds, int kout, int32_t* sel, hipStream_t s);
// MDA per node: sel[v*(q-f) ..] = the rows of node v's least-diameter subset
// of q-f peers (C(q, f) subsets searched by one workgroup), ascending.
hipError_t enqueue_peer_mda(const DistSums& ds, int nodes, const int32_t* peers, int q, int f,
                            int32_t* sel, hipStream_t s);
hipError_t enqueue_mean_nodes(const float* x, int n, int64_t d, int nodes, const int32_t* rows,
                              int k, float* y, hipStream_t s);
hipError_t enqueue_median_nodes(const float* x, int n, int64_t d, int nodes, const int32_t* rows,
                                int k, float* y, hipStream_t s);
hipError_t enqueue_bulyan_nodes(const float* x, int n, int64_t d, int nodes, int q, int f,
                                const int32_t* sel, float* y, hipStream_t s);

// Byzantine rows from the honest ones (byzantine.hip); kinds as garfield_attack.
enum AttackKind { kAttackReverse = 0, kAttackRandom = 1, kAttackLittle = 2, kAttackEmpire = 3 };
hipError_t enqueue_attack(int kind, const float* honest, int h, int64_t d, double param,
                          uint64_t seed, float* byz, int nbyz, hipStream_t s);
// Variance condition: stats[0] = sum_{i<j} D[i][j] / (h (h-1)) over the h rows
// the distance sums `ds` came from, stats[1] = ||grad||^2. Scratch:
// sqnorm_parts(d, grad) fp64 partials.
int64_t sqnorm_parts(int64_t d, const float* grad);
hipError_t enqueue_variance_stats(const DistSums& ds, int h, const float* grad, int64_t d,
                                  double* partial, double* stats, hipStream_t s);

// MDA subset search: C(n, f) at or above mda_cover_min() subsets by vertex
// covers of the "farther than" graphs (one workgroup, no scratch), below it
// by enumeration (scratch: mda_blocks(n, f) x 16 bytes).
int64_t mda_cover_min();
void set_mda_cover_min(int64_t subsets);
bool mda_uses_cover(int n, int f);
int64_t binomial(int a, int b);  // exact, or -1 if above 2^62
int mda_blocks(int n, int f);
size_t mda_scratch_bytes(int n, int f);
hipError_t enqueue_mda_select(const DistSums& ds, int f, void* scratch, int32_t* sel,
                              hipStream_t s);

// Workgroups per CU of the gathering aggregation kernels (aggregate.hip): 0
// (the default) applies each kernel's rule (median and Bulyan's band path
// capped at 2 to 4, the rest uncapped), > 0 caps the median and Bulyan at
// that many, < 0 leaves the residency to the registers.
int stream_residency();
void set_stream_residency(int wgs_per_cu);

// Streaming aggregation kernels over the coordinates.
// Row lists are device int32 arrays (nullptr = rows 0..k-1); an entry outside
// [0, n) is clamped into it, so a bad list cannot make a kernel read outside x.
// Read-rate probe (aggregate.hip): `blocks` workgroups sum the count floats
// at x (16-byte aligned, count % 4 == 0) grid-stride; sums[b] = workgroup b's.
hipError_t enqueue_stream_read(const float* x, int64_t count, int blocks, float* sums,
                               hipStream_t s);
hipError_t enqueue_mean_rows(const float* x, int n, int64_t d, const int32_t* rows, int k,
                             float* out, hipStream_t s);
// The same mean for a selection of k distinct rows (sel, as a selection kernel
// writes it), from the column sums the distance step wrote: the sum of the
// rows not in sel taken from colsum, where colsum is not NaN (the same exact
// value as the rows' sum in listed order), else the rows of sel summed as
// enqueue_mean_rows sums them.
hipError_t enqueue_mean_complement(const float* x, int n, int64_t d, const int32_t* sel, int k,
                                   const double* colsum, float* out, hipStream_t s);
hipError_t enqueue_median(const float* x, int n, int64_t d, const int32_t* rows, int k,
                          float* out, hipStream_t s);
hipError_t enqueue_bulyan_aggregate(const float* x, int n, int f, int64_t d, const int32_t* sel,
                                    float* out, hipStream_t s);

// Width of the register loads of the streaming kernels and the distance
// engines: 4 (16-byte accesses at dword alignment, f4u) for a float-aligned
// pointer, 1 otherwise. Every input the entry points accept is float-aligned
// (check_common), so inputs always get 4; the 1-float paths of the streaming
// kernels serve only an output that is not float-aligned.
int load_width(const float* p);

// Segmented aggregation: acc[i*n + j] += D[i][j] of one segment (all i, j < n;
// the diagonal stays 0), and acc[0 .. count) = 0.
hipError_t enqueue_accumulate_dist(const DistSums& ds, double* acc, hipStream_t s);
hipError_t enqueue_zero_f64(double* p, int count, hipStream_t s);

}  // namespace garfield
