/*
 * garfield.h -- Byzantine-resilient gradient aggregation rules (GARs) on one
 * MI355X (gfx950) GPU.
 *
 * The rules are those of Section 3.1 of "Garfield: System Support for
 * Byzantine Machine Learning" (arXiv:2010.05888): coordinate-wise Median,
 * Krum and Multi-Krum, MDA (minimum-diameter averaging) and Bulyan, plus the
 * plain Average the paper benchmarks them against (Section 6.3).
 *
 * Common conventions for every entry point below:
 *   - x is a DEVICE pointer to n input vectors of d fp32 values, row-major:
 *     vector i occupies x[i*d .. i*d+d-1]. It is only read. It must be
 *     4-byte aligned (as every fp32 allocation is; GARFIELD_EINVAL otherwise).
 *   - out, sel, dist and rows are DEVICE pointers owned by the caller. The
 *     library never frees caller memory and never writes outside the sizes
 *     stated per function.
 *   - stream is a hipStream_t passed as void* (NULL = the default stream). All
 *     work is enqueued on it asynchronously; the call returns once enqueued.
 *     No host<->device copy happens inside any call.
 *   - Arguments are validated on the host before anything is enqueued. On an
 *     error, nothing is enqueued and out/sel/dist are left untouched. No call
 *     aborts or throws across this interface.
 *   - Scratch memory (partial sums, the distance matrix, scores) lives in a
 *     per-device workspace the library allocates on first use and grows when a
 *     call needs more; growing it waits for the device to go idle. Calls on
 *     one device share that workspace, so calls issued on different streams of
 *     the same device must not overlap in time.
 *   - Index outputs (sel) are sets written in ascending order. Ties in a
 *     ranking are broken towards the lower index.
 *   - Preconditions not checked: finite inputs with |x| < FLT_MAX/2, and x,
 *     out, sel, rows, dist valid device allocations of the stated sizes.
 *   - d == 0 is allowed (all distances are 0, so ties pick the lowest
 *     indices; nothing is written to out).
 *   - 1 <= n <= GARFIELD_NMAX.
 */
#ifndef GARFIELD_H
#define GARFIELD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define GARFIELD_NMAX 64
/* Largest number of candidate subsets C(n, f) MDA will enumerate. */
#define GARFIELD_MDA_MAX_SUBSETS 2147483647LL
/* The same per node in a contraction step (C(q, f)). */
#define GARFIELD_CONTRACT_MDA_MAX_SUBSETS 1048576LL

typedef enum garfield_status {
  GARFIELD_OK = 0,
  GARFIELD_EINVAL = 1,  /* null pointer, n < 1, f < 0, d < 0, m or k out of range */
  GARFIELD_EREQ = 2,    /* n below the rule's requirement in f (Section 3.1) */
  GARFIELD_ETOOBIG = 3, /* n > GARFIELD_NMAX, C(n, f) > GARFIELD_MDA_MAX_SUBSETS, or
                           d > (2^31 - 1) * 256 (beyond one launch) */
  GARFIELD_ENOMEM = 4,  /* the workspace could not be allocated */
  GARFIELD_EHIP = 5     /* a HIP call or kernel launch failed */
} garfield_status;

/* Rule identifiers for garfield_workspace_bytes. */
typedef enum garfield_rule {
  GARFIELD_RULE_DIST = 0,
  GARFIELD_RULE_KRUM = 1,
  GARFIELD_RULE_MULTIKRUM = 2,
  GARFIELD_RULE_MEDIAN = 3,
  GARFIELD_RULE_BULYAN = 4,
  GARFIELD_RULE_MDA = 5,
  GARFIELD_RULE_AVERAGE = 6,
  GARFIELD_RULE_MULTIKRUM_ITERATED = 7
} garfield_rule;

/*
 * Pairwise squared Euclidean distances, the distance Krum, MDA and Bulyan
 * score with (Section 3.1 items 2-4):
 *   dist[i*n + j] = sum_c (x[i][c] - x[j][c])^2,  symmetric, zero diagonal.
 * dist: device, n*n fp64. Per-tile partial sums are formed in fp32 and
 * combined across tiles in fp64 in a fixed order, so the result is
 * deterministic and identical input vectors give identical rows of dist.
 */
garfield_status garfield_pairwise_sqdist(const float* x, int n, int64_t d, double* dist,
                                         void* stream);

/*
 * Multi-Krum (Section 3.1 item 2): score(i) = sum of the n-f-2 smallest
 * dist[i][j], j != i; select the m vectors of lowest (score, index) and
 * average them. Requires n >= 2f+3 (else GARFIELD_EREQ) and 1 <= m <= n-f;
 * m <= 0 means the default m = n-f.
 * out: device, d fp32 = mean of the selected vectors, or NULL to compute the
 *      selection only (e.g. to feed garfield_median through `rows`).
 * sel: device, m int32, the selected indices in ascending order.
 * The mean is the fp64 sum of the selected vectors in ascending index order,
 * rounded once to fp32. For n <= 12 with 2m > n + 4 the distance pass also
 * stores each coordinate's fp64 sum over all n vectors (d doubles of
 * workspace), and the mean pass subtracts the n - m others from it wherever
 * every such sum is provably exact (the coordinate's exponents span at most
 * 23 binades), summing the selected vectors elsewhere: the same bits from
 * fewer bytes read.
 * Short inputs (n <= 12, out float-aligned, d up to about 10^5 coordinates)
 * take two launches instead of three or four: the distance pass, then one
 * kernel whose workgroups each add the distance partials, make the selection
 * and write the mean of their 1,024 coordinates -- the same selection and
 * the same bits.
 */
garfield_status garfield_multikrum(const float* x, int n, int f, int64_t d, int m, float* out,
                                   int32_t* sel, void* stream);

/*
 * garfield_multikrum for callers that cannot allocate device memory: code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc. Same arguments, validation, selection and output as
 * garfield_multikrum (the mean always sums the selected vectors; the result is
 * the same bits). Its scratch is a fixed array of
 * GARFIELD_NOALLOC_SCRATCH_BYTES in each device's memory, reserved when the
 * library is loaded and held until the process ends; the call itself
 * allocates and frees nothing (when the opt-in per-kernel timing of
 * garfield_tuning.h is on, its events are created as for every call).
 * Returns GARFIELD_ETOOBIG when the distance step of (n, d) needs more
 * scratch than that: up to about 1.7e8 coordinates at n = 20 and any d that
 * fits in memory for n > 20. Every call on one device uses that device's one
 * array and leaves it holding its own intermediate values: calls that overlap
 * in time on one device (other streams, other threads) race and give wrong
 * results; each call writes every scratch byte it reads before reading it.
 */
#define GARFIELD_NOALLOC_SCRATCH_BYTES (64u << 20)
garfield_status garfield_multikrum_noalloc(const float* x, int n, int f, int64_t d, int m,
                                           float* out, int32_t* sel, void* stream);

/* Krum (Section 3.1 item 2): Multi-Krum with m = 1; out is a copy of vector
 * sel[0]. out may be NULL. */
garfield_status garfield_krum(const float* x, int n, int f, int64_t d, float* out, int32_t* sel,
                              void* stream);

/*
 * Iterated Multi-Krum: Multi-Krum run as repeated Krum, the form Section 4.4
 * names next to Bulyan when it caches distances across iterations. m rounds;
 * each selects the vector of lowest (score, index) among those not yet
 * selected, scoring against the not-yet-selected set with max(r-f-2, 0)
 * neighbours (r = vectors left) -- the selection stage of garfield_bulyan,
 * stopped after m rounds. Then the mean of the m selected vectors, as in
 * garfield_multikrum. Requirements and m as for garfield_multikrum (m = 1 is
 * Krum). The one-shot and the iterated selection can differ once m > 1.
 * out: device, d fp32, or NULL.   sel: device, m int32, ascending.
 */
garfield_status garfield_multikrum_iterated(const float* x, int n, int f, int64_t d, int m,
                                            float* out, int32_t* sel, void* stream);

/*
 * Coordinate-wise median (Section 3.1 item 1) over the k vectors whose
 * indices are listed in `rows` (device int32, each in [0, n)), or over all n
 * vectors when rows is NULL (k is then ignored). Odd k: the middle value,
 * which is one of the inputs bit for bit. Even k: the mean of the two middle
 * values. Requires n >= 2f+1 (f is only checked against n). 1 <= k <= n.
 * out: device, d fp32.
 */
garfield_status garfield_median(const float* x, int n, int f, int64_t d, const int32_t* rows,
                                int k, float* out, void* stream);

/*
 * Bulyan (Section 3.1 item 4) with Krum as the inner rule. theta = n-2f
 * rounds each select the vector of lowest (score, index) among those not yet
 * selected, scoring against the not-yet-selected set with max(r-f-2, 0)
 * neighbours (r = vectors left). Then per coordinate: the median of the theta
 * selected values, and the mean of the beta = theta-2f values closest to it
 * (closeness key (|v - median|, v)). Requires n >= 4f+3.
 * out: device, d fp32.   sel: device, theta int32, ascending.
 */
garfield_status garfield_bulyan(const float* x, int n, int f, int64_t d, float* out,
                                int32_t* sel, void* stream);

/*
 * MDA, minimum-diameter averaging (Section 3.1 item 3): among all subsets of
 * n-f vectors, the first in lexicographic order whose diameter (largest
 * squared distance inside it) is smallest; output its mean. Requires
 * n >= 2f+1 and C(n, f) <= GARFIELD_MDA_MAX_SUBSETS (else GARFIELD_ETOOBIG).
 * out: device, d fp32 (may be NULL).   sel: device, n-f int32, ascending.
 */
garfield_status garfield_mda(const float* x, int n, int f, int64_t d, float* out, int32_t* sel,
                             void* stream);

/* Average, the non-robust baseline rule of the paper's micro-benchmark
 * (Section 6.3): out[c] = (1/n) sum_i x[i][c], summed in fp64. */
garfield_status garfield_average(const float* x, int n, int64_t d, float* out, void* stream);

/*
 * One contraction step for n nodes at once (decentralized learning, Section 5:
 * each node aggregates, with the rule, the vectors it receives from q peers,
 * and repeats). x: device, n x d fp32 row-major, row v = node v's vector.
 * peers: device, n x q int32, row v = the q distinct nodes v hears from (each
 * in [0, n); v itself may be among them). y: device, n x d fp32 (must not
 * overlap x), row v receives rule(x[peers[v][0]], ..., x[peers[v][q-1]]) with
 * f Byzantine vectors tolerated among the q: rule = GARFIELD_RULE_KRUM,
 * _MULTIKRUM, _MULTIKRUM_ITERATED (m as for garfield_multikrum, over q),
 * _BULYAN, _MEDIAN, _MDA or _AVERAGE (others: GARFIELD_EINVAL). The rule's
 * requirement applies to q (e.g. q >= 2f+3 for Krum; GARFIELD_EREQ); MDA
 * also needs C(q, f) <= GARFIELD_CONTRACT_MDA_MAX_SUBSETS, since one
 * workgroup searches a node's subsets (GARFIELD_ETOOBIG). Within a node, ties
 * go to the earlier position in its peer list (for MDA: the first subset of
 * positions in lexicographic order); a mean adds the selected rows in
 * ascending row order (Average: in peer-list order).
 * Distances are computed once for all n rows; selection runs one workgroup
 * per node and aggregation one launch for all nodes. Repeat with x and y
 * swapped for several steps. 1 <= q <= n <= GARFIELD_NMAX.
 */
garfield_status garfield_contract_step(int rule, const float* x, int n, int64_t d,
                                       const int32_t* peers, int q, int f, int m, float* y,
                                       void* stream);

/*
 * Byzantine rows on the device: the attacks Garfield's Byzantine workers and
 * servers implement (Section 3.2, Main objects; Section 6.5 uses random
 * vectors and vectors reversed and amplified by -100). From the h honest
 * vectors `honest` (device, h x d fp32 row-major, read only), write nbyz
 * Byzantine vectors to `byz` (device, nbyz x d fp32 row-major, e.g. the last
 * rows of a rule's input). byz must not overlap honest.
 *   GARFIELD_ATTACK_REVERSE  byz[b] = param * honest[b % h] (param = -100:
 *                            reversed and amplified), the product formed in
 *                            fp64 and rounded once.
 *   GARFIELD_ATTACK_RANDOM   byz[b][c] = param * N(0, 1) (param = the standard
 *                            deviation); honest and h are not used. Normals by
 *                            Box-Muller from Philox4x32-10 (Salmon et al.,
 *                            SC'11) with key = seed and counter (c/4 low and
 *                            high 32 bits, b, 0): words 0-1 give coordinates
 *                            4q and 4q+1, words 2-3 give 4q+2 and 4q+3, each
 *                            word w mapped to ((w >> 9) + 1/2) 2^-23. A value
 *                            depends only on (seed, b, c). fp32 arithmetic.
 *   GARFIELD_ATTACK_LITTLE   "little is enough": byz[b][c] = mean_c - param *
 *                            std_c, over the h honest values of coordinate c
 *                            (population standard deviation), in fp64, rounded
 *                            once; every Byzantine vector is the same.
 *   GARFIELD_ATTACK_EMPIRE   "fall of empires": byz[b][c] = -param * mean_c.
 * Requires 0 <= nbyz <= GARFIELD_NMAX, finite param, and for every kind but
 * RANDOM 1 <= h <= GARFIELD_NMAX.
 */
typedef enum garfield_attack_kind {
  GARFIELD_ATTACK_REVERSE = 0,
  GARFIELD_ATTACK_RANDOM = 1,
  GARFIELD_ATTACK_LITTLE = 2,
  GARFIELD_ATTACK_EMPIRE = 3
} garfield_attack_kind;

garfield_status garfield_attack(int kind, const float* honest, int h, int64_t d, double param,
                                uint64_t seed, float* byz, int nbyz, void* stream);

/*
 * The variance condition of Section 3.1 (Tradeoffs): a rule is safe when
 * kappa * Delta * sigma <= ||grad L|| for some kappa > 1, with sigma^2 =
 * E||g - E g||^2 the variance of an honest gradient estimate.
 *
 * garfield_variance_stats: from h >= 2 honest gradient estimates g (device,
 * h x d fp32 row-major) and the true gradient grad (device, d fp32, e.g.
 * computed on a very large batch), writes stats (device, 2 fp64):
 *   stats[0] = sum_{i<j} ||g_i - g_j||^2 / (h (h-1)), the unbiased estimate of
 *              sigma^2 (equal to sum_i ||g_i - mean||^2 / (h-1)), from the
 *              same distance step the rules use;
 *   stats[1] = ||grad||^2, summed in fp64 in a fixed order.
 * h <= GARFIELD_NMAX.
 *
 * garfield_delta: Delta for rule GARFIELD_RULE_MDA (the paper's minimum-
 * diameter rule: 2 sqrt(2) f / (n-f)), GARFIELD_RULE_KRUM
 * (sqrt(2 (n-f + (f (n-f-2) + f^2 (n-f-1)) / (n-2f-2)))) or
 * GARFIELD_RULE_MEDIAN (sqrt(n-f)); NaN for other rules, n < 1, f < 0, or n
 * below the rule's requirement. Host function.
 * The condition holds for some kappa > 1 iff sqrt(stats[1]) > Delta *
 * sqrt(stats[0]).
 */
garfield_status garfield_variance_stats(const float* g, int h, int64_t d, const float* grad,
                                        double* stats, void* stream);
double garfield_delta(int rule, int n, int f);

/*
 * The condition's margin for rule, n, f from the statistics above, copied to
 * HOST memory by the caller (stats_host[0] = sigma^2, stats_host[1] =
 * ||grad||^2): sqrt(stats_host[1]) / (Delta * sqrt(stats_host[0])); the
 * condition holds for some kappa > 1 iff the margin exceeds 1. +inf when
 * Delta * sigma is 0 (and ||grad|| is not), NaN where garfield_delta is NaN,
 * stats_host is NULL or a statistic is negative or NaN. Host function.
 */
double garfield_variance_margin(int rule, int n, int f, const double* stats_host);

/*
 * Segmented aggregation (per-layer aggregation, Section 4.2). A squared
 * distance is a sum over coordinates, so the distances between the n full
 * vectors are the sums of the distances between their segments (for
 * instance one segment per layer, aggregated as the layers' gradients come
 * in). A segmented aggregation accumulates the segments' distance matrices,
 * makes the rule's one selection from the total, then aggregates every
 * segment with that selection: the result equals the rule applied to the
 * concatenated vectors (the selection up to the rounding of the fp64 sums,
 * the aggregate of each segment exactly as the unsegmented call computes
 * those coordinates).
 *
 *   garfield_seg_create(rule, n, f, m, &seg)   rule: GARFIELD_RULE_KRUM,
 *       _MULTIKRUM or _MULTIKRUM_ITERATED (m as for garfield_multikrum),
 *       _BULYAN, _MDA, _MEDIAN or
 *       _AVERAGE; the requirements of the rule are checked here (EINVAL,
 *       EREQ, ETOOBIG as for the direct calls). Allocates the session's
 *       n x n fp64 running sum and n int32 selection on the current device
 *       (ENOMEM on failure) and waits for the device once. The sum starts at 0.
 *   garfield_seg_accumulate(seg, x, d, stream)   x: device, n x d fp32
 *       row-major, the same segment of each of the n vectors; adds its
 *       distances (a no-op for Median and Average).
 *   garfield_seg_select(seg, sel, stream)   the rule's selection on the sum;
 *       sel: device, the rule's count of int32 (m, n-2f or n-f), ascending,
 *       or NULL to keep it only inside the session (a no-op for Median and
 *       Average).
 *   garfield_seg_aggregate(seg, x, d, out, stream)   aggregates one segment
 *       (n x d, as in accumulate) with the session's selection into out
 *       (device, d fp32). EINVAL before the first select after a reset.
 *   garfield_seg_reset(seg, stream)   zeroes the sum for the next step.
 *   garfield_seg_destroy(seg)   waits for the session's device, frees it.
 *
 * All enqueued work goes on `stream` in call order; a session must not be
 * used from two streams at once, and it shares the per-device workspace with
 * every other call (see above).
 */
typedef struct garfield_segmented garfield_segmented;

garfield_status garfield_seg_create(int rule, int n, int f, int m, garfield_segmented** out);
garfield_status garfield_seg_reset(garfield_segmented* seg, void* stream);
garfield_status garfield_seg_accumulate(garfield_segmented* seg, const float* x, int64_t d,
                                        void* stream);
garfield_status garfield_seg_select(garfield_segmented* seg, int32_t* sel, void* stream);
garfield_status garfield_seg_aggregate(garfield_segmented* seg, const float* x, int64_t d,
                                       float* out, void* stream);
garfield_status garfield_seg_destroy(garfield_segmented* seg);

/*
 * Segment tables: the same session fed with vectors stored apart, K segments
 * at a time. ptrs (DEVICE, K*n pointers): ptrs[s*n + i] points to segment s of
 * vector i, dims[s] fp32 values (HOST array of K lengths, each >= 0; every
 * pointer 4-byte aligned). Typical uses: each worker's per-layer gradients
 * (K = number of layers), or n whole vectors in separate buffers (K = 1, the
 * row-pointer form of every rule: create, accumulate_table, select,
 * aggregate_table).
 *   garfield_seg_accumulate_table(seg, ptrs, dims, K, stream)   adds the
 *       distances of all K segments; one launch per 96 segments, whatever
 *       their sizes, instead of one distance step per segment.
 *   garfield_seg_aggregate_table(seg, ptrs, dims, K, outs, stream)   aggregates
 *       every segment with the session's selection; outs (HOST array of K
 *       DEVICE pointers, each to dims[s] fp32 values, 4-byte aligned).
 * Distances: the direct engine for n <= 20, else the Gram engine over the
 * table (one reference row, probed on the longest segment, for every
 * segment). Results equal those of garfield_seg_accumulate /
 * garfield_seg_aggregate on the same segments held as n x d matrices for
 * n <= 20 (whatever the engine threshold); for n > 20 the distances differ
 * from the matrix sessions' only by rounding (the Gram engine's bound). A
 * launch takes at most 2^31 - 1 workgroups or stages (GARFIELD_ETOOBIG).
 */
garfield_status garfield_seg_accumulate_table(garfield_segmented* seg, const float* const* ptrs,
                                              const int64_t* dims, int K, void* stream);
garfield_status garfield_seg_aggregate_table(garfield_segmented* seg, const float* const* ptrs,
                                             const int64_t* dims, int K, float* const* outs,
                                             void* stream);

/*
 * Bytes of workspace one call of `rule` with these sizes uses (0 if the
 * arguments are invalid). Informational: the library allocates it itself.
 */
size_t garfield_workspace_bytes(int rule, int n, int f, int64_t d, int m);

/* Free the workspace of the current device (waits for the device first). */
garfield_status garfield_release(void);

/* Static, human-readable description of a status code. */
const char* garfield_strerror(garfield_status s);

/* Library version string, e.g. "garfield-mi355x 0.1". */
const char* garfield_version(void);

#ifdef __cplusplus
}
#endif

#endif /* GARFIELD_H */
