"""CPU oracle for the Garfield aggregation rules (test infrastructure only).

Only the test suite, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package. The product path (the HIP library and its
Python binding) never touches it, and the two share no code.

``garfield_oracle.cpp`` is the fp64 C++/OpenMP implementation of each rule as
Section 3.1 of the paper defines it; this module only marshals numpy arrays to
it. ``bruteforce.py`` is an independent exact-rational implementation used to
pin the oracle on tiny inputs.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "garfield_oracle.cpp")
_LIB = os.path.join(_HERE, "libgarfield_oracle.so")

OK, EINVAL, EREQ = 0, 1, 2


def build(force: bool = True) -> str:
    """Compile the oracle with g++ (no fast-math: sums keep their order)."""
    if force or not os.path.exists(_LIB):
        cmd = ["g++", "-O2", "-std=c++17", "-fopenmp", "-fPIC", "-shared",
               "-Wall", "-Wextra", "-o", _LIB + ".tmp", _SRC]
        subprocess.run(cmd, check=True)
        os.replace(_LIB + ".tmp", _LIB)
    return _LIB


_lib = None


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=False)
        lib = ctypes.CDLL(_LIB)
        f32p = ctypes.POINTER(ctypes.c_float)
        f64p = ctypes.POINTER(ctypes.c_double)
        i32p = ctypes.POINTER(ctypes.c_int32)
        i64p = ctypes.POINTER(ctypes.c_int64)
        c_int, c_i64 = ctypes.c_int, ctypes.c_int64
        lib.oracle_pairwise_sqdist.argtypes = [f32p, c_int, c_i64, f64p]
        lib.oracle_krum_scores.argtypes = [f32p, c_int, c_int, c_i64, f64p]
        lib.oracle_multikrum.argtypes = [f32p, c_int, c_int, c_i64, c_int, f32p, i32p, f64p, f64p]
        lib.oracle_median.argtypes = [f32p, c_int, c_int, c_i64, i32p, c_int, f32p]
        lib.oracle_bulyan.argtypes = [f32p, c_int, c_int, c_i64, f32p, i32p, i32p, f64p, f64p]
        lib.oracle_multikrum_iterated.argtypes = [f32p, c_int, c_int, c_i64, c_int, f32p, i32p,
                                                  i32p, f64p, f64p]
        u32p = ctypes.POINTER(ctypes.c_uint32)
        lib.oracle_philox4x32_10.argtypes = [u32p, u32p, u32p]
        lib.oracle_philox4x32_10.restype = None
        lib.oracle_attack.argtypes = [c_int, f32p, c_int, c_i64, ctypes.c_double, ctypes.c_uint64,
                                      f32p, c_int]
        lib.oracle_variance_stats.argtypes = [f32p, c_int, c_i64, f32p, f64p]
        lib.oracle_mda.argtypes = [f32p, c_int, c_int, c_i64, f32p, i32p, f64p, f64p, i64p, f64p]
        for fn in (lib.oracle_pairwise_sqdist, lib.oracle_krum_scores, lib.oracle_multikrum,
                   lib.oracle_median, lib.oracle_bulyan, lib.oracle_mda,
                   lib.oracle_multikrum_iterated, lib.oracle_attack, lib.oracle_variance_stats):
            fn.restype = ctypes.c_int
        lib.oracle_omp_team_size.argtypes = []
        lib.oracle_omp_team_size.restype = ctypes.c_int
        _lib = lib
    return _lib


def omp_team_size() -> int:
    """Threads in the OpenMP team the oracle's parallel loops use on this host."""
    return int(_load().oracle_omp_team_size())


class OracleError(ValueError):
    def __init__(self, code: int, what: str):
        super().__init__(f"{what}: oracle status {code}")
        self.code = code


def _ptr(a, ctype):
    if a is None:
        return None
    return a.ctypes.data_as(ctypes.POINTER(ctype))


def _rows(x):
    x = np.ascontiguousarray(x, dtype=np.float32)
    if x.ndim != 2:
        raise ValueError("expected an n x d array")
    return x


def _check(code, what):
    if code != OK:
        raise OracleError(code, what)


def pairwise_sqdist(x) -> np.ndarray:
    """n x n fp64 matrix of squared Euclidean distances."""
    x = _rows(x)
    n, d = x.shape
    D = np.zeros((n, n), dtype=np.float64)
    _check(_load().oracle_pairwise_sqdist(_ptr(x, ctypes.c_float), n, d,
                                          _ptr(D, ctypes.c_double)), "pairwise_sqdist")
    return D


def krum_scores(x, f: int) -> np.ndarray:
    x = _rows(x)
    n, d = x.shape
    s = np.zeros(n, dtype=np.float64)
    _check(_load().oracle_krum_scores(_ptr(x, ctypes.c_float), n, f, d,
                                      _ptr(s, ctypes.c_double)), "krum_scores")
    return s


def multikrum(x, f: int, m: int | None = None, return_scores: bool = False,
              return_distances: bool = False):
    """(aggregate fp32 [d], sel int32 [m] ascending[, scores fp64 [n]][, D fp64 [n, n]])."""
    x = _rows(x)
    n, d = x.shape
    mm = (n - f) if (m is None or m <= 0) else m
    out = np.zeros(d, dtype=np.float32)
    sel = np.zeros(max(mm, 1), dtype=np.int32)
    scores = np.zeros(n, dtype=np.float64)
    D = np.zeros((n, n), dtype=np.float64)
    _check(_load().oracle_multikrum(_ptr(x, ctypes.c_float), n, f, d, 0 if m is None else m,
                                    _ptr(out, ctypes.c_float), _ptr(sel, ctypes.c_int32),
                                    _ptr(scores, ctypes.c_double), _ptr(D, ctypes.c_double)),
           "multikrum")
    res = (out, sel[:mm])
    if return_scores:
        res += (scores,)
    if return_distances:
        res += (D,)
    return res


def multikrum_iterated(x, f: int, m: int | None = None, return_rounds: bool = False,
                       return_distances: bool = False):
    """(aggregate, sel [m] ascending[, picks in order, round scores m x n][, D])."""
    x = _rows(x)
    n, d = x.shape
    mm = (n - f) if (m is None or m <= 0) else m
    out = np.zeros(d, dtype=np.float32)
    sel = np.zeros(max(mm, 1), dtype=np.int32)
    picks = np.zeros(max(mm, 1), dtype=np.int32)
    rs = np.zeros((max(mm, 1), n), dtype=np.float64)
    D = np.zeros((n, n), dtype=np.float64)
    _check(_load().oracle_multikrum_iterated(_ptr(x, ctypes.c_float), n, f, d,
                                             0 if m is None else m, _ptr(out, ctypes.c_float),
                                             _ptr(sel, ctypes.c_int32),
                                             _ptr(picks, ctypes.c_int32),
                                             _ptr(rs, ctypes.c_double), _ptr(D, ctypes.c_double)),
           "multikrum_iterated")
    res = (out, sel[:mm])
    if return_rounds:
        res += (picks[:mm], rs[:mm])
    if return_distances:
        res += (D,)
    return res


def krum(x, f: int, return_scores: bool = False):
    return multikrum(x, f, 1, return_scores)


def median(x, f: int = 0, rows=None) -> np.ndarray:
    x = _rows(x)
    n, d = x.shape
    out = np.zeros(d, dtype=np.float32)
    if rows is None:
        code = _load().oracle_median(_ptr(x, ctypes.c_float), n, f, d, None, n,
                                     _ptr(out, ctypes.c_float))
    else:
        r = np.ascontiguousarray(rows, dtype=np.int32)
        code = _load().oracle_median(_ptr(x, ctypes.c_float), n, f, d,
                                     _ptr(r, ctypes.c_int32), len(r), _ptr(out, ctypes.c_float))
    _check(code, "median")
    return out


def bulyan(x, f: int, return_rounds: bool = False, return_distances: bool = False):
    """(aggregate, sel ascending[, picks in order, round scores theta x n][, D])."""
    x = _rows(x)
    n, d = x.shape
    theta = n - 2 * f
    out = np.zeros(d, dtype=np.float32)
    sel = np.zeros(max(theta, 1), dtype=np.int32)
    picks = np.zeros(max(theta, 1), dtype=np.int32)
    rs = np.zeros((max(theta, 1), n), dtype=np.float64)
    D = np.zeros((n, n), dtype=np.float64)
    _check(_load().oracle_bulyan(_ptr(x, ctypes.c_float), n, f, d, _ptr(out, ctypes.c_float),
                                 _ptr(sel, ctypes.c_int32), _ptr(picks, ctypes.c_int32),
                                 _ptr(rs, ctypes.c_double), _ptr(D, ctypes.c_double)), "bulyan")
    res = (out, sel[:theta])
    if return_rounds:
        res += (picks[:theta], rs[:theta])
    if return_distances:
        res += (D,)
    return res


def mda(x, f: int, return_diameters: bool = False, return_distances: bool = False):
    """(aggregate, sel ascending[, best diameter, next larger diameter, #subsets at best][, D])."""
    x = _rows(x)
    n, d = x.shape
    out = np.zeros(d, dtype=np.float32)
    sel = np.zeros(max(n - f, 1), dtype=np.int32)
    best = np.zeros(1, dtype=np.float64)
    second = np.zeros(1, dtype=np.float64)
    nbest = np.zeros(1, dtype=np.int64)
    D = np.zeros((n, n), dtype=np.float64)
    _check(_load().oracle_mda(_ptr(x, ctypes.c_float), n, f, d, _ptr(out, ctypes.c_float),
                              _ptr(sel, ctypes.c_int32), _ptr(best, ctypes.c_double),
                              _ptr(second, ctypes.c_double), _ptr(nbest, ctypes.c_int64),
                              _ptr(D, ctypes.c_double)), "mda")
    res = (out, sel[:n - f])
    if return_diameters:
        res += (float(best[0]), float(second[0]), int(nbest[0]))
    if return_distances:
        res += (D,)
    return res


# --- Byzantine vectors and the variance condition ----------------------------------

ATTACKS = {"reverse": 0, "random": 1, "little": 2, "empire": 3}


def philox4x32_10(ctr, key):
    """The four output words of Philox4x32-10 for a counter (4 words) and key (2)."""
    c = np.ascontiguousarray(ctr, dtype=np.uint32)
    k = np.ascontiguousarray(key, dtype=np.uint32)
    out = np.zeros(4, dtype=np.uint32)
    _load().oracle_philox4x32_10(_ptr(c, ctypes.c_uint32), _ptr(k, ctypes.c_uint32),
                                 _ptr(out, ctypes.c_uint32))
    return out.tolist()


def attack(kind: str, honest, nbyz: int, param: float, seed: int = 0, d: int | None = None):
    """nbyz x d fp32 Byzantine vectors (reading R9 of the oracle's header)."""
    if honest is None:
        h, dd, hp = 0, int(d), None
    else:
        honest = _rows(honest)
        h, dd = honest.shape
        hp = _ptr(honest, ctypes.c_float)
    out = np.zeros((nbyz, dd), dtype=np.float32)
    _check(_load().oracle_attack(ATTACKS[kind], hp, h, dd, float(param),
                                 seed & 0xFFFFFFFFFFFFFFFF, _ptr(out, ctypes.c_float), nbyz),
           "attack")
    return out


def variance_stats(g, grad):
    """[sum_i ||g_i - mean||^2 / (h - 1), ||grad||^2] in fp64 (reading R10)."""
    g = _rows(g)
    h, d = g.shape
    t = np.ascontiguousarray(grad, dtype=np.float32).reshape(-1)
    stats = np.zeros(2, dtype=np.float64)
    _check(_load().oracle_variance_stats(_ptr(g, ctypes.c_float), h, d, _ptr(t, ctypes.c_float),
                                         _ptr(stats, ctypes.c_double)), "variance_stats")
    return stats


def delta(rule: str, n: int, f: int) -> float:
    """Delta of the variance condition (Section 3.1, Tradeoffs): the minimum-
    diameter rule 2 sqrt(2) f / (n - f), Krum sqrt(2 (n - f + (f (n - f - 2) +
    f^2 (n - f - 1)) / (n - 2f - 2))), Median sqrt(n - f); NaN for other rules
    or n below the rule's requirement (2f+1, 2f+3, 2f+1)."""
    import math

    if n < 1 or f < 0:
        return math.nan
    if rule == "mda":
        return 2.0 * math.sqrt(2.0) * f / (n - f) if n >= 2 * f + 1 else math.nan
    if rule == "krum":
        if n < 2 * f + 3:
            return math.nan
        return math.sqrt(2.0 * ((n - f) + (f * (n - f - 2) + f * f * (n - f - 1)) / (n - 2 * f - 2)))
    if rule == "median":
        return math.sqrt(n - f) if n >= 2 * f + 1 else math.nan
    return math.nan


# --- contraction steps ----------------------------------------------------------

def contract_step(rule: str, x, peers, f: int, m: int | None = None):
    """Row v = `rule` applied to the rows peers[v] of x, in peer-list order
    (ties in a selection go to the earlier position in the list): the rule
    functions above on each node's gathered rows. Average adds the rows in list
    order in fp64 and rounds once. Returns (y, selections as sorted row
    indices, or None)."""
    x = _rows(x)
    peers = np.asarray(peers, dtype=np.int64)
    y = np.zeros_like(x)
    sels = []
    for v in range(x.shape[0]):
        xs = np.ascontiguousarray(x[peers[v]])
        if rule == "average":
            acc = np.zeros(x.shape[1], dtype=np.float64)
            for r in range(xs.shape[0]):
                acc += xs[r].astype(np.float64)
            y[v] = (acc / xs.shape[0]).astype(np.float32)
            continue
        if rule == "median":
            y[v] = median(xs, f)
            continue
        fn = {"krum": lambda a: multikrum(a, f, 1), "multikrum": lambda a: multikrum(a, f, m),
              "multikrum_iterated": lambda a: multikrum_iterated(a, f, m),
              "bulyan": lambda a: bulyan(a, f), "mda": lambda a: mda(a, f)}[rule]
        out, sel = fn(xs)[:2]
        y[v] = out
        sels.append(sorted(int(peers[v][t]) for t in sel))
    return y, (sels if sels else None)
