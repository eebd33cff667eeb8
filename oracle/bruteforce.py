"""Exact brute-force reference for tiny inputs (test infrastructure only).

Everything here is computed with ``fractions.Fraction`` and by enumeration,
with formulations that differ on purpose from the fp64 oracle so that the two
pin each other:

* a Krum score is the minimum, over all k-subsets of the other vectors, of the
  summed squared distances (instead of sorting and taking a prefix);
* Multi-Krum's set is the m-subset whose sorted (score, index) list is
  lexicographically smallest;
* a median is found by counting (an element with at most (k-1)/2 values
  strictly below and at most (k-1)/2 strictly above it) instead of sorting;
* Bulyan's beta closest values are the beta-subset (by position) whose sorted
  key list is lexicographically smallest;
* MDA enumerates every (n-f)-subset;
* iterated Multi-Krum repeats the subset-minimum Krum score over the rows
  left, like Bulyan's selection here.

Definitions follow Section 3.1 of the paper (items 1-4); the readings taken
where it is silent are the same as the fp64 oracle's (see its header).
Inputs are sequences of rows of numbers convertible to Fraction.
"""
from __future__ import annotations

from fractions import Fraction
from itertools import combinations


def _rows(x):
    return [[Fraction(v) for v in row] for row in x]


def sqdist(a, b) -> Fraction:
    return sum(((p - q) * (p - q) for p, q in zip(a, b)), Fraction(0))


def distance_matrix(x):
    x = _rows(x)
    n = len(x)
    return [[sqdist(x[i], x[j]) for j in range(n)] for i in range(n)]


def krum_score(D, cand, i, k) -> Fraction:
    others = [j for j in cand if j != i]
    k = min(k, len(others))
    if k <= 0:
        return Fraction(0)
    return min(sum((D[i][j] for j in sub), Fraction(0)) for sub in combinations(others, k))


def mean(x, rows):
    x = _rows(x)
    d = len(x[0]) if x else 0
    return [sum((x[i][c] for i in rows), Fraction(0)) / len(rows) for c in range(d)]


def multikrum(x, f, m=None):
    """Returns (aggregate, sel ascending, scores) exactly."""
    n = len(x)
    if n < 2 * f + 3:
        raise ValueError("Multi-Krum requires n >= 2f+3")
    m = n - f if (m is None or m <= 0) else m
    if m > n - f:
        raise ValueError("m out of range")
    D = distance_matrix(x)
    scores = [krum_score(D, range(n), i, n - f - 2) for i in range(n)]
    best = min(combinations(range(n), m), key=lambda sub: sorted((scores[i], i) for i in sub))
    sel = sorted(best)
    return mean(x, sel), sel, scores


def krum(x, f):
    return multikrum(x, f, 1)


def median_of(vals):
    """Middle order statistic by counting; even counts average the two middles."""
    k = len(vals)

    def is_order_stat(v, r):  # v is the r-th smallest (0-based) of vals
        below = sum(1 for w in vals if w < v)
        equal = sum(1 for w in vals if w == v)
        return below <= r < below + equal

    def order_stat(r):
        return next(v for v in vals if is_order_stat(v, r))

    if k % 2 == 1:
        return order_stat((k - 1) // 2)
    return (order_stat(k // 2 - 1) + order_stat(k // 2)) / 2


def median(x, f=0, rows=None):
    n = len(x)
    if n < 2 * f + 1:
        raise ValueError("Median requires n >= 2f+1")
    x = _rows(x)
    rows = list(range(n)) if rows is None else list(rows)
    d = len(x[0])
    return [median_of([x[i][c] for i in rows]) for c in range(d)]


def bulyan(x, f):
    """Returns (aggregate, sel ascending, picks in order) exactly."""
    n = len(x)
    if n < 4 * f + 3:
        raise ValueError("Bulyan requires n >= 4f+3")
    theta, beta = n - 2 * f, n - 4 * f
    D = distance_matrix(x)
    remaining = list(range(n))
    picks = []
    for _ in range(theta):
        k = max(len(remaining) - f - 2, 0)
        scored = [(krum_score(D, remaining, i, k), i) for i in remaining]
        _, w = min(scored)
        picks.append(w)
        remaining.remove(w)
    xr = _rows(x)
    out = []
    for c in range(len(xr[0])):
        vals = [xr[i][c] for i in picks]
        med = median_of(vals)
        keys = [(abs(v - med), v) for v in vals]
        best = min(combinations(range(theta), beta), key=lambda sub: sorted(keys[t] for t in sub))
        out.append(sum((vals[t] for t in best), Fraction(0)) / beta)
    return out, sorted(picks), picks


def multikrum_iterated(x, f, m=None):
    """Returns (aggregate, sel ascending, picks in order) exactly: m rounds,
    each taking the lowest (score, index) over the rows left, scored against
    the rows left with max(r - f - 2, 0) neighbours."""
    n = len(x)
    if n < 2 * f + 3:
        raise ValueError("Multi-Krum requires n >= 2f+3")
    m = n - f if (m is None or m <= 0) else m
    D = distance_matrix(x)
    remaining = list(range(n))
    picks = []
    for _ in range(m):
        k = max(len(remaining) - f - 2, 0)
        _, w = min((krum_score(D, remaining, i, k), i) for i in remaining)
        picks.append(w)
        remaining.remove(w)
    return mean(x, picks), sorted(picks), picks


def mda(x, f):
    """Returns (aggregate, sel ascending, diameter) exactly."""
    n = len(x)
    if n < 2 * f + 1:
        raise ValueError("MDA requires n >= 2f+1")
    D = distance_matrix(x)
    best, best_diam = None, None
    for sub in combinations(range(n), n - f):  # lexicographic order
        diam = max((D[i][j] for i, j in combinations(sub, 2)), default=Fraction(0))
        if best_diam is None or diam < best_diam:
            best, best_diam = list(sub), diam
    return mean(x, best), best, best_diam
