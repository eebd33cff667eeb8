"""Tolerances and decision-gap checks for GPU-vs-oracle parity.

Distances. The library's D differs from the oracle's fp64 D only by fp32
rounding inside a tile (everything across tiles is fp64). Per entry:

* direct engine: each lane adds at most 16 squares (kDirectLaneCoords) into
  an fp32 accumulator with one fused multiply-add each, after one rounded
  fp32 subtraction; for positive terms that is a relative error of at most
  (16 + 2) u, u = 2^-24.
* Gram engine: y = fl(x - x_ref) is rounded once (|error| <= u |y|), and each
  row's y over a stage of 256 coordinates (counted from the start of the
  vector, or of each segment of a segment table) is rounded to a multiple of
  2^-k, k = min(21 - E, 127) with E the exponent of the stage's largest |y|
  (-126 when that is 0 or subnormal): an error of at most 2^-k / 2. With
  e_i = || u |y_i| + 2^-k / 2 || (over all coordinates), the products of the
  quantized values are exact, so the stage sums are the exact Gram entries of
  the quantized rows and D~_ij = ||y~_i - y~_j||^2 exactly, up to the fp64
  accumulation: |D~_ij - D_ij| <= 2 sqrt(D_ij) (e_i + e_j) + (e_i + e_j)^2.
  The fp64 sums over stages and tiles and the final G_ii + G_jj - 2 G_ij add
  at most (S + 1203) 2^-53 * 2 (N~_i + N~_j), S the number of stages,
  N~_i = (sqrt(N_i) + e_i)^2 and N_i = ||x_i - x_ref||^2 (the oracle's
  D[i][ref]).

Gram reference row. The Gram engine shifts every row by one input row, chosen
by a probe over a sample of the coordinates: 4 runs of 256 consecutive
coordinates starting at r * (d // 4), r = 0..3 (all of d when d <= 1024). The
probe distance of (i, j) is the squared distance over the sample; a row's
score is the sum of its ceil(n/2) smallest probe distances (itself included,
at 0), and the reference is the lowest (score, index). The library sums each
coordinate's square in fp32 (at most 4 per lane, after one rounded
subtraction) before fp64, a relative error of at most (4 + 2) u per probe
distance. gram_reference_rule() evaluates the rule from the oracle's fp64
distances on the same sample, so the tests check the library's pick against
it instead of trusting it.

Decisions. A selection is "pinned" when every decision it makes is separated
by more than the summed error bounds of the two quantities compared, so any
D within those bounds makes the same decision; identical input rows are
exact ties on both sides (broken by the lower index), and are not gaps.
"""
from __future__ import annotations

from itertools import combinations

import numpy as np

U = 2.0 ** -24
DIRECT_LANE_COORDS = 16
EPS_DIRECT = (DIRECT_LANE_COORDS + 2) * U
GRAM_STAGE = 256


PROBE_RUNS = 4
PROBE_RUN = 256
EPS_PROBE = 6 * U + 1e-12


def probe_columns(d):
    """Coordinates the Gram engine's probe reads."""
    if d <= PROBE_RUNS * PROBE_RUN:
        return [np.arange(d)]
    return [np.arange(r * (d // PROBE_RUNS), r * (d // PROBE_RUNS) + PROBE_RUN)
            for r in range(PROBE_RUNS)]


def gram_reference_rule(x):
    """(best, candidates): the reference row the probe rule picks on the oracle's
    exact probe distances, and every row whose score interval, under the
    library's probe error, reaches the best one's (the library's pick must be
    among them; when that set is {best} the pick is pinned)."""
    import oracle

    x = np.asarray(x, dtype=np.float32)
    n, d = x.shape
    xs = np.ascontiguousarray(x[:, np.concatenate(probe_columns(d))]) if d else x
    P = np.zeros((n, n))
    for cols in probe_columns(d):
        P += oracle.pairwise_sqdist(np.ascontiguousarray(x[:, cols]))
    h = (n + 1) // 2
    score = np.array([np.sort(P[i])[:h].sum() for i in range(n)])
    lo = np.array([np.sort(P[i] * (1 - EPS_PROBE))[:h].sum() for i in range(n)])
    hi = np.array([np.sort(P[i])[:h].sum() * (1 + EPS_PROBE) for i in range(n)])
    best = int(min(range(n), key=lambda i: (score[i], i)))
    # rows equal on the sample have bit-identical probe rows: an exact tie,
    # which goes to the lower index
    same = [i for i in range(n) if np.array_equal(xs[i], xs[best])]
    cands = sorted(i for i in range(n) if lo[i] <= hi[best] and i not in same[1:])
    if best not in cands:
        cands = sorted(cands + [best])
    return best, cands


def checked_reference(x, ref, byzantine=()):
    """Assert that the library's reference row `ref` follows the probe rule on x
    (equal to the rule's pick when that is pinned, else one of the rows the
    error bound cannot separate from it; identical rows tie to the lower
    index) and is not a Byzantine row; return it."""
    best, cands = gram_reference_rule(x)
    assert ref in cands, ("Gram reference row", ref, "rule", best, "candidates", cands)
    if cands == [best]:
        assert ref == best, ("Gram reference row", ref, "rule", best)
    assert ref not in set(int(b) for b in byzantine), ("Byzantine reference row", ref, byzantine)
    return ref


def agg_close(got, want):
    """North-star aggregate tolerance: max(1e-5 |want|, 1e-6) per coordinate."""
    got = np.asarray(got, dtype=np.float64)
    want = np.asarray(want, dtype=np.float64)
    tol = np.maximum(1e-5 * np.abs(want), 1e-6)
    err = np.abs(got - want)
    bad = np.nonzero(err > tol)[0]
    return bad.size == 0, (int(bad[0]) if bad.size else -1), float(err.max(initial=0.0))


def gram_error_norms(x, ref, segments=None):
    """(e, stages): per row, the 2-norm over all coordinates of the bound on the
    Gram engine's per-coordinate error u |y| + 2^-k / 2 (y = fl(x - x_ref),
    k per row and stage as the kernel chooses it), and the number of stages.
    `segments`: lengths of the consecutive segments whose stages start anew
    (a segment table); default one segment of all of x."""
    x = np.asarray(x, dtype=np.float32)
    n, d = x.shape
    segments = [d] if segments is None else list(segments)
    assert sum(segments) == d
    e2 = np.zeros(n)
    stages = 0
    xr = x[ref]
    start = 0
    for length in segments:
        if length == 0:
            continue
        S = -(-length // GRAM_STAGE)
        stages += S
        for i in range(n):
            y = np.abs(x[i, start:start + length] - xr[start:start + length])  # fp32, as the kernel
            pad = np.zeros(S * GRAM_STAGE, dtype=np.float32)
            pad[:length] = y
            st = pad.reshape(S, GRAM_STAGE)
            mx = st.max(axis=1)
            _, ex = np.frexp(mx)
            E = np.where(mx < np.float32(2.0 ** -126), -126, ex.astype(np.int64) - 1)
            k = np.minimum(21 - E, 127)
            half = np.ldexp(1.0, -k - 1)[:, None]        # per stage
            eps = U * st.astype(np.float64) + half        # padding: |y| = 0, counted as 0
            eps[-1, length - (S - 1) * GRAM_STAGE:] = 0.0
            e2[i] += float((eps * eps).sum())
        start += length
    return np.sqrt(e2), stages


def dist_bounds(D, engine, ref=None, x=None, segments=None):
    """n x n absolute error bounds on the library's D entries, from the oracle's
    D (and, for the Gram engine, the input x and the reference row `ref`, which
    set the quantization steps; segments as in gram_error_norms)."""
    n = D.shape[0]
    if engine == "direct":
        B = EPS_DIRECT * D
    elif engine == "gram":
        assert x is not None and ref is not None
        e, stages = gram_error_norms(x, ref, segments)
        N = D[:, ref]
        Nq = (np.sqrt(N) + e) ** 2
        es = e[:, None] + e[None, :]
        fp64 = (stages + 1203) * 2.0 ** -53 * 2.0 * (Nq[:, None] + Nq[None, :])
        B = (2.0 * np.sqrt(D) * es + es * es + fp64) * (1.0 + 1e-9)
    else:  # no distance kernel ran: D is exactly 0
        B = np.zeros_like(D)
    B = B + 1e-300
    B[np.arange(n), np.arange(n)] = 0.0
    return B


def identical_rows(D):
    """Rows i, j are identical iff the oracle's exact-difference D[i][j] is 0."""
    return D == 0.0


def _score_intervals(D, B, cand, k):
    """Interval [lo, hi] holding the library's Krum score of each candidate.

    With N_i the oracle's k nearest of i among cand, the library sums its own
    k smallest perturbed distances, which is at most sum_{j in N_i} (D+B) and
    at least the sum of the k smallest (D-B).
    """
    out = {}
    for i in cand:
        others = [j for j in cand if j != i]
        near = sorted(others, key=lambda j: (D[i, j], j))[:k]
        hi = float(sum(D[i, j] + B[i, j] for j in near))
        lo = float(sum(sorted(D[i, j] - B[i, j] for j in others)[:k]))
        out[i] = (lo, hi, near)
    return out


def _structural_tie(D, B, a, b, k, cand, same):
    """Oracle scores of a and b are equal, and so are the library's."""
    if same[a, b] or k == 0:
        return True
    if k != 1:
        return False
    # mutual nearest neighbours: both scores are the one entry D[a][b], which
    # the library stores symmetrically; it must be clearly the nearest of each
    for i, j in ((a, b), (b, a)):
        rest = [D[i, t] - B[i, t] for t in cand if t not in (i, j)]
        if rest and D[i, j] + B[i, j] >= min(rest):
            return False
    return True


def _pair_margin(sc, iv, a, b, D, B, k, cand, same):
    """Margin by which a (ranked first) is decided before b."""
    if sc[a] == sc[b]:
        return np.inf if _structural_tie(D, B, a, b, k, cand, same) else -np.inf
    return iv[b][0] - iv[a][1]


def krum_pinned(scores, D, B, f, m, same):
    """Multi-Krum's selected set is decided beyond the error bounds."""
    n = len(scores)
    k = n - f - 2
    order = sorted(range(n), key=lambda i: (scores[i], i))
    chosen, rest = order[:m], order[m:]
    iv = _score_intervals(D, B, range(n), k)
    margin = np.inf
    for a in chosen:
        for b in rest:
            margin = min(margin, _pair_margin(scores, iv, a, b, D, B, k, range(n), same))
    return margin > 0, margin


def bulyan_pinned(picks, round_scores, D, B, n, f, same):
    remaining = list(range(n))
    margin = np.inf
    for r, w in enumerate(picks):
        k = max(len(remaining) - f - 2, 0)
        s = round_scores[r]
        iv = _score_intervals(D, B, remaining, k)
        for j in remaining:
            if j == w:
                continue
            margin = min(margin, _pair_margin(s, iv, w, j, D, B, k, remaining, same))
        remaining.remove(w)
    return margin > 0, margin


def mda_pinned(D, B, n, f, best_set):
    """The lexicographically first minimum-diameter subset is decided beyond the bounds."""
    s = n - f
    best_set = tuple(int(i) for i in best_set)

    def interval(S):
        pairs = list(combinations(S, 2))
        if not pairs:
            return 0.0, 0.0, None
        lo = max(D[i, j] - B[i, j] for i, j in pairs)
        hi = max(D[i, j] + B[i, j] for i, j in pairs)
        top = max(pairs, key=lambda p: D[p])
        return lo, hi, top

    _, best_hi, best_top = interval(best_set)
    best = max((D[i, j] for i, j in combinations(best_set, 2)), default=0.0)
    margin = np.inf
    for S in combinations(range(n), s):
        if S == best_set:
            continue
        diam = max((D[i, j] for i, j in combinations(S, 2)), default=0.0)
        lo, hi, top = interval(S)
        if diam > best:
            margin = min(margin, lo - best_hi)
        elif diam == best and S < best_set:
            return False, -np.inf  # oracle would not have picked best_set
        elif diam == best:
            # an exact tie: both must have the same, clearly largest, pair
            for T, t in ((S, top), (best_set, best_top)):
                rest = [D[i, j] + B[i, j] for i, j in combinations(T, 2) if (i, j) != t]
                if t != best_top or (rest and max(rest) >= D[t] - B[t]):
                    return False, -np.inf
    return margin > 0, margin
