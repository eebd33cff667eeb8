"""Pins for the CPU oracle (no GPU).

The paper prints no numeric example of any rule, so the oracle is pinned by:
hand-worked examples (tests/golden), an independent exact-rational brute force
on thousands of tiny integer inputs (where fp64 arithmetic is exact, so the two
must agree bit for bit, ties included), library routines for the special
cases that have one (scipy's squared Euclidean distances, numpy's median and
mean), closed forms (f = 0 reduces Multi-Krum with m = n, Bulyan and MDA to the
mean) and invariants (permutation, identical inputs, exact power-of-two
scaling, negation).
"""
import json
import os
from fractions import Fraction

import numpy as np
import pytest
from scipy.spatial.distance import cdist

import oracle
from oracle import bruteforce as bf

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "worked_examples.json")


def _f32(fr):
    return np.float32(float(Fraction(fr)))


def _examples():
    with open(GOLDEN) as fh:
        return json.load(fh)["examples"]


@pytest.mark.parametrize("ex", _examples(), ids=lambda e: e["name"])
def test_bruteforce_matches_hand_worked(ex):
    x = ex["x"]
    k = ex["krum"]
    out, sel, scores = bf.krum(x, k["f"])
    assert [str(s) for s in scores] == k["scores"]
    assert sel == k["sel"] and [str(v) for v in out] == k["out"]
    for mk in ex["multikrum"]:
        out, sel, _ = bf.multikrum(x, mk["f"], mk["m"])
        assert sel == mk["sel"] and [str(v) for v in out] == mk["out"]
    assert [str(v) for v in bf.median(x, ex["median"]["f"])] == ex["median"]["out"]
    for md in ex["mda"]:
        out, sel, diam = bf.mda(x, md["f"])
        assert sel == md["sel"] and str(diam) == md["diameter"]
        assert [str(v) for v in out] == md["out"]
    for bu in ex["bulyan"]:
        out, sel, picks = bf.bulyan(x, bu["f"])
        assert sel == bu["sel"] and [str(v) for v in out] == bu["out"]
        if "picks" in bu:
            assert picks == bu["picks"]
    for mi in ex.get("multikrum_iterated", []):
        out, sel, picks = bf.multikrum_iterated(x, mi["f"], mi["m"])
        assert sel == mi["sel"] and picks == mi["picks"]
        assert [str(v) for v in out] == mi["out"]


@pytest.mark.parametrize("ex", _examples(), ids=lambda e: e["name"])
def test_oracle_matches_hand_worked(ex):
    x = np.array(ex["x"], dtype=np.float32)
    k = ex["krum"]
    out, sel, scores = oracle.krum(x, k["f"], return_scores=True)
    assert scores.tolist() == [float(Fraction(s)) for s in k["scores"]]
    assert sel.tolist() == k["sel"]
    assert out.tolist() == [_f32(v) for v in k["out"]]
    for mk in ex["multikrum"]:
        out, sel = oracle.multikrum(x, mk["f"], mk["m"])
        assert sel.tolist() == mk["sel"] and out.tolist() == [_f32(v) for v in mk["out"]]
    assert oracle.median(x, ex["median"]["f"]).tolist() == [_f32(v) for v in ex["median"]["out"]]
    for md in ex["mda"]:
        out, sel, best, _, _ = oracle.mda(x, md["f"], return_diameters=True)
        assert sel.tolist() == md["sel"] and best == float(Fraction(md["diameter"]))
        assert out.tolist() == [_f32(v) for v in md["out"]]
    for bu in ex["bulyan"]:
        out, sel, picks, _ = oracle.bulyan(x, bu["f"], return_rounds=True)
        assert sel.tolist() == bu["sel"] and out.tolist() == [_f32(v) for v in bu["out"]]
        if "picks" in bu:
            assert picks.tolist() == bu["picks"]
    for mi in ex.get("multikrum_iterated", []):
        out, sel, picks, _ = oracle.multikrum_iterated(x, mi["f"], mi["m"], return_rounds=True)
        assert sel.tolist() == mi["sel"] and picks.tolist() == mi["picks"]
        assert out.tolist() == [_f32(v) for v in mi["out"]]


def _tiny_cases(seed, count):
    """Small-integer inputs (fp64 arithmetic on them is exact), with planted
    duplicate rows so that exact ties are common."""
    rng = np.random.default_rng(seed)
    for _ in range(count):
        n = int(rng.integers(1, 10))
        d = int(rng.integers(1, 4))
        x = rng.integers(-6, 7, size=(n, d)).astype(np.float32)
        if n >= 3 and rng.random() < 0.4:
            x[rng.integers(0, n)] = x[rng.integers(0, n)]
        yield x


def _check_against_bf(x):
    n = x.shape[0]
    xl = x.astype(int).tolist()
    for f in range(0, n):
        if n >= 2 * f + 3:
            for m in sorted({1, n - f, max(1, (n - f) // 2)}):
                ob, sb, scb = bf.multikrum(xl, f, m)
                oo, so, sco = oracle.multikrum(x, f, m, return_scores=True)
                assert so.tolist() == sb, (x, f, m)
                assert sco.tolist() == [float(s) for s in scb]
                assert oo.tolist() == [_f32(v) for v in ob], (x, f, m)
                ob, sb, pb = bf.multikrum_iterated(xl, f, m)
                oo, so, po, _ = oracle.multikrum_iterated(x, f, m, return_rounds=True)
                assert so.tolist() == sb and po.tolist() == pb, (x, f, m)
                assert oo.tolist() == [_f32(v) for v in ob], (x, f, m)
        if n >= 2 * f + 1:
            assert oracle.median(x, f).tolist() == [_f32(v) for v in bf.median(xl, f)], (x, f)
            ob, sb, db = bf.mda(xl, f)
            oo, so, do, _, _ = oracle.mda(x, f, return_diameters=True)
            assert so.tolist() == sb and do == float(db), (x, f)
            assert oo.tolist() == [_f32(v) for v in ob], (x, f)
        if n >= 4 * f + 3:
            ob, sb, pb = bf.bulyan(xl, f)
            oo, so, po, _ = oracle.bulyan(x, f, return_rounds=True)
            assert so.tolist() == sb and po.tolist() == pb, (x, f)
            assert oo.tolist() == [_f32(v) for v in ob], (x, f)


@pytest.mark.parametrize("seed", range(8))
def test_oracle_equals_bruteforce_on_tiny_integer_inputs(seed):
    for x in _tiny_cases(1000 + seed, 60):
        _check_against_bf(x)


def test_oracle_median_subset_equals_bruteforce():
    rng = np.random.default_rng(7)
    for _ in range(200):
        n = int(rng.integers(1, 12))
        x = rng.integers(-5, 6, size=(n, 3)).astype(np.float32)
        k = int(rng.integers(1, n + 1))
        rows = rng.choice(n, size=k, replace=False)
        got = oracle.median(x, 0, rows=rows)
        want = bf.median(x.astype(int).tolist(), 0, rows=rows.tolist())
        assert got.tolist() == [_f32(v) for v in want]


# --- library routines and closed forms -------------------------------------------

def test_distances_equal_scipy_sqeuclidean():
    rng = np.random.default_rng(3)
    for n, d in [(1, 5), (2, 1), (7, 1000), (13, 257), (64, 300)]:
        x = rng.standard_normal((n, d)).astype(np.float32)
        want = cdist(x.astype(np.float64), x.astype(np.float64), "sqeuclidean")
        got = oracle.pairwise_sqdist(x)
        np.testing.assert_allclose(got, want, rtol=1e-12, atol=0)
        assert np.all(np.diag(got) == 0) and np.array_equal(got, got.T)


@pytest.mark.parametrize("k", [1, 2, 3, 4, 7, 10, 49, 64])
def test_median_equals_numpy_median(k):
    rng = np.random.default_rng(k)
    x = rng.standard_normal((k, 501)).astype(np.float32)
    want = np.median(x.astype(np.float64), axis=0).astype(np.float32)
    got = oracle.median(x, 0)
    assert np.array_equal(got, want)
    if k % 2 == 1:  # an odd median is one of the inputs
        assert np.all(np.any(x == got[None, :], axis=0))


def test_median_of_three_is_med3():
    rng = np.random.default_rng(5)
    x = rng.standard_normal((3, 1000)).astype(np.float32)
    med3 = np.maximum(np.minimum(x[0], x[1]), np.minimum(np.maximum(x[0], x[1]), x[2]))
    assert np.array_equal(oracle.median(x, 1), med3)


@pytest.mark.parametrize("n", [3, 5, 8, 17])
def test_f_zero_rules_reduce_to_the_mean(n):
    rng = np.random.default_rng(n)
    x = rng.standard_normal((n, 333)).astype(np.float32)
    mean = x.astype(np.float64).mean(axis=0)
    out, sel = oracle.multikrum(x, 0, n)
    assert sel.tolist() == list(range(n))
    np.testing.assert_allclose(out, mean, rtol=1e-6, atol=1e-7)
    out, sel = oracle.bulyan(x, 0)
    assert sel.tolist() == list(range(n))
    np.testing.assert_allclose(out, mean, rtol=1e-6, atol=1e-7)
    out, sel = oracle.mda(x, 0)
    assert sel.tolist() == list(range(n))
    np.testing.assert_allclose(out, mean, rtol=1e-6, atol=1e-7)
    out, sel = oracle.multikrum_iterated(x, 0, n)
    assert sel.tolist() == list(range(n))
    np.testing.assert_allclose(out, mean, rtol=1e-6, atol=1e-7)


def test_iterated_multikrum_m1_is_krum_and_theta_rounds_are_bulyans_picks():
    rng = np.random.default_rng(12)
    for n, f in [(5, 1), (7, 1), (11, 2), (19, 4)]:
        x = rng.standard_normal((n, 64)).astype(np.float32)
        o1, s1 = oracle.multikrum_iterated(x, f, 1)
        o2, s2 = oracle.krum(x, f)
        assert s1.tolist() == s2.tolist() and np.array_equal(o1, o2)
        if n >= 4 * f + 3:
            _, sel, picks, _ = oracle.multikrum_iterated(x, f, n - 2 * f, return_rounds=True)
            _, bsel, bpicks, _ = oracle.bulyan(x, f, return_rounds=True)
            assert picks.tolist() == bpicks.tolist() and sel.tolist() == bsel.tolist()


def test_multikrum_m1_is_krum_and_krum_returns_an_input():
    rng = np.random.default_rng(11)
    for n, f in [(5, 1), (7, 2), (11, 4), (20, 3)]:
        x = rng.standard_normal((n, 64)).astype(np.float32)
        o1, s1 = oracle.multikrum(x, f, 1)
        o2, s2 = oracle.krum(x, f)
        assert s1.tolist() == s2.tolist() and np.array_equal(o1, o2)
        assert np.array_equal(o2, x[s2[0]])


# --- invariants ----------------------------------------------------------------

def _all_rules(x, f):
    n = x.shape[0]
    res = {}
    if n >= 2 * f + 3:
        res["krum"] = oracle.krum(x, f)
        res["multikrum"] = oracle.multikrum(x, f)
        res["multikrum_iterated"] = oracle.multikrum_iterated(x, f)
    if n >= 2 * f + 1:
        res["median"] = (oracle.median(x, f), None)
        res["mda"] = oracle.mda(x, f)
    if n >= 4 * f + 3:
        res["bulyan"] = oracle.bulyan(x, f)
    return res


@pytest.mark.parametrize("n,f", [(7, 1), (11, 2), (10, 2), (15, 3)])
def test_permutation_invariance(n, f):
    rng = np.random.default_rng(100 + n)
    x = rng.standard_normal((n, 97)).astype(np.float32)
    x[: n - f] *= 0.1  # honest cluster, f outliers
    perm = rng.permutation(n)
    a, b = _all_rules(x, f), _all_rules(x[perm], f)
    for name in a:
        if name == "bulyan" and f < 3:
            # Bulyan's last round runs Krum on 2f+1 vectors with f-1 neighbours:
            # for f = 1 every score is 0 and for f = 2 the closest pair always
            # ties, so the lower index decides and row order matters.
            continue
        if name == "multikrum_iterated":
            # its last two rounds (m = n-f) score with 0 neighbours, so the
            # lower index decides there as well
            continue
        np.testing.assert_allclose(b[name][0], a[name][0], rtol=1e-6, atol=1e-7, err_msg=name)
        if a[name][1] is not None:
            assert sorted(perm[b[name][1]].tolist()) == a[name][1].tolist(), name


def test_identical_inputs_return_that_input():
    rng = np.random.default_rng(9)
    row = rng.standard_normal(50).astype(np.float32)
    for n in [1, 3, 7, 11]:
        x = np.tile(row, (n, 1))
        for f in range(0, n):
            for name, (out, _) in _all_rules(x, f).items():
                assert np.array_equal(out, row), (n, f, name)


def test_power_of_two_scaling_is_exact():
    rng = np.random.default_rng(13)
    x = rng.standard_normal((11, 200)).astype(np.float32)
    a, b = _all_rules(x, 2), _all_rules(x * np.float32(8.0), 2)
    for name in a:
        assert np.array_equal(b[name][0], a[name][0] * np.float32(8.0)), name
        if a[name][1] is not None:
            assert np.array_equal(b[name][1], a[name][1]), name


def test_negation():
    rng = np.random.default_rng(17)
    x = rng.standard_normal((11, 200)).astype(np.float32)
    a, b = _all_rules(x, 2), _all_rules(-x, 2)
    for name in a:  # no ties in continuous data, so every rule is odd in x
        assert np.array_equal(b[name][0], -a[name][0]), name
        if a[name][1] is not None:
            assert np.array_equal(b[name][1], a[name][1]), name


# --- requirements on n and f (Section 3.1) ---------------------------------------

def test_requirements_are_enforced():
    x = np.zeros((6, 4), dtype=np.float32)
    with pytest.raises(oracle.OracleError) as e:
        oracle.krum(x, 2)  # needs n >= 2f+3 = 7
    assert e.value.code == oracle.EREQ
    with pytest.raises(oracle.OracleError) as e:
        oracle.bulyan(x, 1)  # needs n >= 4f+3 = 7
    assert e.value.code == oracle.EREQ
    with pytest.raises(oracle.OracleError) as e:
        oracle.median(x, 3)  # needs n >= 2f+1 = 7
    assert e.value.code == oracle.EREQ
    with pytest.raises(oracle.OracleError) as e:
        oracle.mda(x, 3)
    assert e.value.code == oracle.EREQ
    with pytest.raises(oracle.OracleError) as e:
        oracle.multikrum(x, 1, 6)  # m <= n-f = 5
    assert e.value.code == oracle.EINVAL
    with pytest.raises(oracle.OracleError) as e:
        oracle.multikrum_iterated(x, 2)  # needs n >= 2f+3 = 7
    assert e.value.code == oracle.EREQ
    with pytest.raises(oracle.OracleError) as e:
        oracle.multikrum_iterated(x, 1, 6)
    assert e.value.code == oracle.EINVAL
    # at the bound every rule runs
    oracle.krum(np.zeros((7, 4), np.float32), 2)
    oracle.bulyan(np.zeros((7, 4), np.float32), 1)
    oracle.median(np.zeros((7, 4), np.float32), 3)
    oracle.mda(np.zeros((7, 4), np.float32), 3)


def test_empty_dimension_selects_lowest_indices():
    x = np.zeros((7, 0), dtype=np.float32)
    out, sel = oracle.multikrum(x, 1, 3)
    assert sel.tolist() == [0, 1, 2] and out.size == 0
    out, sel = oracle.multikrum_iterated(x, 1, 3)
    assert sel.tolist() == [0, 1, 2] and out.size == 0
    out, sel = oracle.mda(x, 2)
    assert sel.tolist() == [0, 1, 2, 3, 4]
    out, sel = oracle.bulyan(x, 1)
    assert sel.tolist() == [0, 1, 2, 3, 4]
