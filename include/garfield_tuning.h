/*
 * garfield_tuning.h -- engine selection knobs of libgarfield, for tests and
 * benchmarks. Results do not depend on them beyond floating-point rounding of
 * the distance matrix; indices and aggregates keep the guarantees stated in
 * garfield.h.
 */
#ifndef GARFIELD_TUNING_H
#define GARFIELD_TUNING_H

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

/*
 * Largest n for which pairwise distances use the direct-difference VALU
 * engine; above it they use the MFMA Gram engine (Y = X - x_ref quantized per
 * 256-coordinate stage, exact int8 MFMA).
 * Valid range 1..GARFIELD_DIRECT_MAX_N_LIMIT (1 means: always MFMA for
 * n >= 2). Returns the previous value, or -1 (and changes nothing) if the
 * value is out of range. Process-wide; not synchronised with calls in flight.
 */
#define GARFIELD_DIRECT_MAX_N_LIMIT 20
#define GARFIELD_DIRECT_MAX_N_DEFAULT 20
int garfield_tuning_set_direct_max_n(int n);

/*
 * Whether garfield_krum and garfield_multikrum (and the no-allocation
 * variant) may make the selection and the mean in one kernel on short inputs:
 * n <= 12 rows, a float-aligned out, the distance pass in at most 256 tiles,
 * and at most 8 MiB of distance partials read again by the combined kernel
 * (each of its workgroups, one per 1,024 coordinates, adds all of them): d up
 * to about 228,000 at n = 7 and 129,000 at n = 12. The combined kernel makes the same selection and
 * writes the same bits as the separate selection and mean kernels. on = 0
 * turns it off; 1 (the default) allows it. Returns the previous setting.
 * Process-wide; not synchronised with calls in flight.
 */
int garfield_tuning_set_fused(int on);

/*
 * MDA's search: from this many candidate subsets C(n, f) on (default 2^20),
 * the least diameter and the lexicographically first subset attaining it are
 * found through vertex covers of the graph of pairs farther apart than a
 * threshold (one workgroup; work grows with 2^f, not with C(n, f)); below it
 * every subset is enumerated. Both give the same subset. Returns the previous
 * value; a negative argument changes nothing. Process-wide; not synchronised
 * with calls in flight.
 */
long long garfield_tuning_set_mda_cover_min(long long subsets);

/*
 * Workgroups per compute unit of the gathering aggregation kernels, capped by
 * reserving LDS the kernels do not use: fewer loads in flight stream faster
 * from HBM. 0 (the default) applies each kernel's own rule -- the median's
 * 16-byte path and Bulyan's beta = 3 path take two to four workgroups per CU
 * (about 100 to 140 KB of loads in flight per CU), the other gathers no cap;
 * a positive value caps the median and Bulyan at that many; a negative one
 * removes every cap. Results do not depend on it. Returns the
 * previous setting. Process-wide; not synchronised with calls in flight.
 */
int garfield_tuning_set_stream_residency(int wgs_per_cu);

/* Engine the distance step would use for (n, d): 0 none (n < 2 or d == 0),
 * 1 direct differences (VALU), 2 Gram (exact integer MFMA). */
int garfield_tuning_distance_engine(int n, long long d);

/* The reference row the Gram engine would shift the n x d device input x by
 * (the row with the smallest sum of its ceil(n/2) nearest probe distances).
 * Enqueues the probe on `stream`, waits for it and returns the index, or -1
 * on error. Lets tests bound the Gram engine's cancellation error. */
int garfield_tuning_gram_reference(const float* x, int n, long long d, void* stream);

/* The same for a segment table of n vectors (ptrs: DEVICE, K*n pointers;
 * dims: HOST, K lengths, as garfield_seg_accumulate_table takes them) with
 * n > 20, whose Gram engine probes the longest segment (the first of equal
 * ones). Returns -1 on error or when every segment is empty. */
int garfield_tuning_table_gram_reference(const float* const* ptrs, int n, const long long* dims,
                                         int K, void* stream);

/*
 * Per-kernel timing. While on, every kernel a call launches is launched with
 * a pair of HIP events that the runtime stamps at the start and the end of
 * that kernel's own dispatch (hipExtLaunchKernelGGL), on the call's stream.
 * Turning it on or off (either way) waits for the device and drops the
 * records collected so far. Returns the previous setting.
 */
int garfield_tuning_set_kernel_timing(int on);

/*
 * Waits for every recorded event and writes one line per kernel name,
 * "name launches total_ms\n", in first-launch order, into buf (host memory,
 * NUL-terminated, truncated to len-1 bytes). Returns the full length.
 */
size_t garfield_tuning_kernel_timing(char* buf, size_t len);

/*
 * Plain streaming read, the yardstick the aggregation kernels' bandwidth is
 * read against: GARFIELD_TUNING_READ_BLOCKS workgroups of 256 lanes walk the
 * `count` fp32 values at x (device) grid-stride, each lane with four 16-byte
 * nontemporal loads in flight, and write each workgroup's fp32 sum to
 * sums[0 .. GARFIELD_TUNING_READ_BLOCKS-1] (device). x must be 16-byte
 * aligned and count a multiple of 4 (else GARFIELD_EINVAL and nothing is
 * enqueued). Asynchronous on `stream`; returns a garfield_status.
 */
#define GARFIELD_TUNING_READ_BLOCKS 512
int garfield_tuning_stream_read(const float* x, long long count, float* sums, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* GARFIELD_TUNING_H */
