"""Generate branch-free selection networks for the per-coordinate kernels.

The coordinate-wise median (Section 3.1 item 1) and Bulyan's trimmed mean
(item 4) need, for every coordinate, the order statistics of k values. On a
64-wide wavefront the cheapest way to get them without divergence is a fixed
network of min/max operations applied to k registers per lane.

Construction: a sorting network on the next power of two N >= k -- Batcher's
odd-even merge sort or Parberry's pairwise sorting network, whichever prunes
to fewer operations -- with the N-k padding wires fixed to -inf (bottom) or
+inf (top). A comparator whose outcome is known from the padding is resolved
at generation time (it becomes a wire rename or disappears). The network is
then pruned backwards from the outputs that are needed: a comparator whose
max (or min) output is never read emits only the other half. Every split of
the padding between -inf and +inf is tried and the cheapest network kept.
Both base networks have the same comparators in number, but the pairwise
one reaches the middle ranks through fewer of them, so it prunes better for
medians (590 -> 512 operations at k = 49).

Each emitted operation is one of
    ("ce", a, b)   v[a], v[b] = min(v[a], v[b]), max(v[a], v[b])
    ("min", a, b)  v[a] = min(v[a], v[b])
    ("max", a, b)  v[b] = max(v[a], v[b])
on the k real registers (after the renames). ``apply_ops`` simulates a list on
numpy arrays; the CPU tests use it to check every network with the 0-1
principle.
"""
from __future__ import annotations

import functools
import os
import sys

NMAX = 64


def _oddeven_merge_sort(n):
    """Comparator list (i, j), i < j, of Batcher's odd-even merge sort on n = 2^p wires."""
    ops = []

    def merge(lo, hi, r):
        step = r * 2
        if step < hi - lo:
            merge(lo, hi, step)
            merge(lo + r, hi, step)
            for i in range(lo + r, hi - r, step):
                ops.append((i, i + r))
        else:
            ops.append((lo, lo + r))

    def sort(lo, hi):
        if hi - lo >= 1:
            mid = lo + (hi - lo) // 2
            sort(lo, mid)
            sort(mid + 1, hi)
            merge(lo, hi, 1)

    sort(0, n - 1)
    return ops


def _pairwise_sort(n):
    """Comparator list (i, j), i < j, of Parberry's pairwise sorting network on
    n = 2^p wires: first every pair (b - a, b) of the blocks of width a = 1, 2,
    4, ... is compared (sorting the pairs, then the pairs of pairs, and so on),
    then a merging phase compares wires d*a apart for shrinking a and d."""
    ops = []
    a = 1
    while a < n:
        b, c = a, 0
        while b < n:
            ops.append((b - a, b))
            b += 1
            c = (c + 1) % a
            if c == 0:
                b += a
        a *= 2
    a //= 4
    e = 1
    while a > 0:
        d = e
        while d > 0:
            b, c = (d + 1) * a, 0
            while b < n:
                ops.append((b - d * a, b))
                b += 1
                c = (c + 1) % a
                if c == 0:
                    b += a
            d //= 2
        a //= 2
        e = e * 2 + 1
    return ops


BASES = {"oddeven": _oddeven_merge_sort, "pairwise": _pairwise_sort}


def _build(k, n_neg, outputs_rank, base="oddeven"):
    """Network for k values padded with n_neg -inf wires below and the rest +inf above.

    outputs_rank: ranks (0-based, among the k real values) that must be exact.
    Returns (ops, out_reg) where out_reg[r] is the register holding rank r.
    """
    n = 1
    while n < k:
        n *= 2
    n_pos = n - k - n_neg
    # wire state: ("neg",), ("pos",) or ("reg", r) -- which register a wire holds
    wire = [None] * n
    for w in range(n_neg):
        wire[w] = ("neg",)
    for r in range(k):
        wire[n_neg + r] = ("reg", r)
    for w in range(n_neg + k, n):
        wire[w] = ("pos",)
    raw = []  # resolved comparators on registers: (lo_reg, hi_reg) meaning lo<-min, hi<-max
    for (i, j) in BASES[base](n):
        a, b = wire[i], wire[j]
        if a[0] == "neg" or b[0] == "pos":
            continue  # already ordered
        if a[0] == "pos" or b[0] == "neg":
            wire[i], wire[j] = b, a  # known swap: a rename
            continue
        raw.append((a[1], b[1]))  # register a[1] receives min, b[1] receives max
    # after sorting, wire n_neg + r holds rank r
    out_reg = {}
    for r in outputs_rank:
        w = wire[n_neg + r]
        assert w[0] == "reg"
        out_reg[r] = w[1]
    # backward liveness pruning
    live = set(out_reg.values())
    ops = []
    for (lo, hi) in reversed(raw):
        need_lo, need_hi = lo in live, hi in live
        if need_lo and need_hi:
            ops.append(("ce", lo, hi))
        elif need_lo:
            ops.append(("min", lo, hi))
        elif need_hi:
            ops.append(("max", lo, hi))
        else:
            continue
        live.add(lo)
        live.add(hi)
    ops.reverse()
    del n_pos
    return ops, out_reg


def _cost(ops):
    return sum(2 if op[0] == "ce" else 1 for op in ops)


def band3_ranks(k):
    """The ranks Bulyan's trimmed mean can use when beta = 3 (the smallest
    theta, n = 4f + 3): odd k, the median c = (k-1)//2 and two on each side;
    even k (median between c-1 and c, c = k//2), c-3 .. c+2. Clipped to 0..k-1."""
    if k % 2:
        c = (k - 1) // 2
        lo, hi = c - 2, c + 2
    else:
        c = k // 2
        lo, hi = c - 3, c + 2
    return list(range(max(lo, 0), min(hi, k - 1) + 1))


@functools.lru_cache(maxsize=None)
def network(k, kind):
    """kind 'median': ranks (k-1)//2 (odd k) or k//2-1, k//2 (even k); 'sort': all ranks;
    'band3': band3_ranks(k)."""
    if kind == "median":
        ranks = [(k - 1) // 2] if k % 2 else [k // 2 - 1, k // 2]
    elif kind == "sort":
        ranks = list(range(k))
    elif kind == "band3":
        ranks = band3_ranks(k)
    else:
        raise ValueError(kind)
    n = 1
    while n < k:
        n *= 2
    best = None
    for base in ("oddeven", "pairwise"):
        for n_neg in range(0, n - k + 1):
            ops, out = _build(k, n_neg, ranks, base)
            if best is None or _cost(ops) < _cost(best[0]):
                best = (ops, out)
    return best


def apply_ops(ops, v):
    """Apply a network to v (list of numpy arrays, one per register), in place."""
    import numpy as np

    for op, a, b in ops:
        if op == "ce":
            lo, hi = np.minimum(v[a], v[b]), np.maximum(v[a], v[b])
            v[a], v[b] = lo, hi
        elif op == "min":
            v[a] = np.minimum(v[a], v[b])
        else:
            v[b] = np.maximum(v[a], v[b])
    return v


def _emit_body(ops):
    lines = []
    for op, a, b in ops:
        if op == "ce":
            lines.append(f"    {{ const float t = v[{a}]; v[{a}] = fmin_(t, v[{b}]); v[{b}] = fmax_(t, v[{b}]); }}")
        elif op == "min":
            lines.append(f"    v[{a}] = fmin_(v[{a}], v[{b}]);")
        else:
            lines.append(f"    v[{b}] = fmax_(v[{a}], v[{b}]);")
    return "\n".join(lines)


def emit_header(nmax=NMAX):
    out = [
        "// Generated by gen_networks.py -- do not edit.",
        "// Branch-free selection networks on k registers (odd-even merge or",
        "// pairwise sorting networks padded to a power of two, resolved and pruned",
        "// at generation time).",
        "#pragma once",
        "",
        "template <int K> struct MedianNet;  // run(): median rank(s) land in v[LO], v[HI]",
        "template <int K> struct SortNet;    // run(): v[R[r]] holds rank r",
        "template <int K> struct BandNet;    // run(): v[reg(r)] holds rank r, FIRST <= r <= LAST",
        "",
    ]
    for k in range(1, nmax + 1):
        ops, reg = network(k, "median")
        ranks = sorted(reg)
        lo, hi = reg[ranks[0]], reg[ranks[-1]]
        out.append(f"template <> struct MedianNet<{k}> {{")
        out.append(f"  static constexpr int LO = {lo}, HI = {hi}, OPS = {_cost(ops)};")
        out.append("  __device__ __forceinline__ static void run(float* v) {")
        body = _emit_body(ops)
        if body:
            out.append(body)
        else:
            out.append("    (void)v;")
        out.append("  }")
        out.append("};")
        ops, reg = network(k, "sort")
        order = ", ".join(str(reg[r]) for r in range(k))
        out.append(f"template <> struct SortNet<{k}> {{")
        out.append(f"  static constexpr int OPS = {_cost(ops)};")
        out.append(f"  __device__ __forceinline__ static int reg(int r) {{ constexpr int R[{k}] = {{{order}}}; return R[r]; }}")
        out.append("  __device__ __forceinline__ static void run(float* v) {")
        body = _emit_body(ops)
        out.append(body if body else "    (void)v;")
        out.append("  }")
        out.append("};")
        ops, reg = network(k, "band3")
        ranks = band3_ranks(k)
        order = ", ".join(str(reg[r]) for r in ranks)
        out.append(f"template <> struct BandNet<{k}> {{")
        out.append(f"  static constexpr int FIRST = {ranks[0]}, LAST = {ranks[-1]}, OPS = {_cost(ops)};")
        out.append(f"  __device__ __forceinline__ static constexpr int reg(int r) {{ constexpr int R[{len(ranks)}] = {{{order}}}; return R[r - FIRST]; }}")
        out.append("  __device__ __forceinline__ static void run(float* v) {")
        body = _emit_body(ops)
        out.append(body if body else "    (void)v;")
        out.append("  }")
        out.append("};")
        out.append("")
    return "\n".join(out) + "\n"


def write_header(path=None, nmax=NMAX):
    path = path or os.path.join(os.path.dirname(os.path.abspath(__file__)), "networks.inc")
    text = emit_header(nmax)
    old = None
    if os.path.exists(path):
        with open(path) as fh:
            old = fh.read()
    if old != text:
        with open(path, "w") as fh:
            fh.write(text)
    return path


if __name__ == "__main__":
    print(write_header(sys.argv[1] if len(sys.argv) > 1 else None))
