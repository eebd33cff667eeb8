"""The generated selection networks are correct (no GPU).

A comparator network sorts (or selects ranks of) every input iff it does so for
every 0/1 input (the 0-1 principle), so for k <= 18 every 0/1 pattern is
checked. Larger k are checked on random 0/1 patterns and random permutations.
"""
import importlib.util
import os

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
_spec = importlib.util.spec_from_file_location(
    "gen_networks", os.path.join(ROOT, "paper_2010_05888_amd", "csrc", "gen_networks.py"))
gen = importlib.util.module_from_spec(_spec)
_spec.loader.exec_module(gen)


def _all_binary(k):
    idx = np.arange(2 ** k, dtype=np.int64)
    return [((idx >> b) & 1).astype(np.float32) for b in range(k)]


def _random_inputs(k, rng, count=20000):
    bins = [rng.integers(0, 2, count).astype(np.float32) for _ in range(k)]
    perms = np.argsort(rng.random((count, k)), axis=1).astype(np.float32)
    return bins, [perms[:, r].copy() for r in range(k)]


def _check(k, kind, cols):
    ops, reg = gen.network(k, kind)
    v = gen.apply_ops(ops, [c.copy() for c in cols])
    ref = np.sort(np.stack(cols, axis=1), axis=1)
    for r, g in reg.items():
        assert np.array_equal(v[g], ref[:, r]), (k, kind, r)


@pytest.mark.parametrize("k", range(1, 19))
@pytest.mark.parametrize("kind", ["median", "sort", "band3"])
def test_network_zero_one_exhaustive(k, kind):
    _check(k, kind, _all_binary(k))


@pytest.mark.parametrize("k", range(19, gen.NMAX + 1))
@pytest.mark.parametrize("kind", ["median", "sort", "band3"])
def test_network_random(k, kind):
    rng = np.random.default_rng(k)
    bins, perms = _random_inputs(k, rng)
    _check(k, kind, bins)
    _check(k, kind, perms)


def test_median_ranks_and_register_map():
    for k in range(1, gen.NMAX + 1):
        _, reg = gen.network(k, "median")
        want = [(k - 1) // 2] if k % 2 else [k // 2 - 1, k // 2]
        assert sorted(reg) == want
        _, reg = gen.network(k, "sort")
        assert sorted(reg) == list(range(k)) and sorted(reg.values()) == list(range(k))
        # the band holds every rank a beta = 3 trimmed mean can take around the median
        _, reg = gen.network(k, "band3")
        c = (k - 1) // 2 if k % 2 else k // 2
        want = range(max(c - 2, 0), min(c + 2, k - 1) + 1) if k % 2 else \
            range(max(c - 3, 0), min(c + 2, k - 1) + 1)
        assert sorted(reg) == list(want)


def test_header_generation_is_deterministic(tmp_path):
    p1 = gen.write_header(str(tmp_path / "a.inc"), nmax=12)
    p2 = gen.write_header(str(tmp_path / "b.inc"), nmax=12)
    assert open(p1).read() == open(p2).read()


@pytest.mark.parametrize("base", sorted(gen.BASES))
@pytest.mark.parametrize("p", range(1, 7))
def test_base_networks_sort(base, p):
    # both base networks sort every 0/1 input (all of them up to 16 wires,
    # 2^17 random ones above) and have Batcher's comparator count,
    # (p^2 - p + 4) 2^(p-2) - 1 for n = 2^p wires
    n = 2 ** p
    cmps = gen.BASES[base](n)
    assert len(cmps) == (p * p - p + 4) * 2 ** p // 4 - 1
    assert all(0 <= i < j < n for i, j in cmps)
    if n <= 16:
        cols = _all_binary(n)
    else:
        rng = np.random.default_rng(n)
        cols = [rng.integers(0, 2, 1 << 17).astype(np.float32) for _ in range(n)]
    for i, j in cmps:
        cols[i], cols[j] = np.minimum(cols[i], cols[j]), np.maximum(cols[i], cols[j])
    a = np.stack(cols, axis=1)
    assert np.all(a[:, :-1] <= a[:, 1:])


def test_pairwise_prunes_the_large_medians():
    # the generator keeps the cheaper base: the k = 49 median needs 512 operations
    ops, _ = gen.network(49, "median")
    assert gen._cost(ops) == 512
