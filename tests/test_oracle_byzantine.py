"""Pins for the oracle's Byzantine vectors and variance condition (no GPU).

Philox4x32-10 is pinned to its published known-answer vectors; the normals
drawn from it to the normal distribution (Kolmogorov-Smirnov) and to their
independence across rows; the moment attacks and the variance estimate to
hand-worked values and to numpy's mean, std and var; Delta to its closed forms
evaluated by hand (tests/golden/byzantine_examples.json).
"""
import json
import math
import os

import numpy as np
import pytest
from scipy import stats as sps

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "byzantine_examples.json")


def _golden():
    with open(GOLDEN) as fh:
        return json.load(fh)


@pytest.mark.parametrize("case", _golden()["philox"], ids=lambda c: c["ctr"][0])
def test_philox_known_answers(case):
    ctr = [int(v, 16) for v in case["ctr"]]
    key = [int(v, 16) for v in case["key"]]
    assert oracle.philox4x32_10(ctr, key) == [int(v, 16) for v in case["out"]]


def test_random_rows_are_standard_normal_and_independent():
    d = 200_003
    z = oracle.attack("random", None, 3, 1.0, seed=12345, d=d).astype(np.float64)
    for b in range(3):
        assert sps.kstest(z[b], "norm").pvalue > 1e-3, b
        assert abs(z[b].mean()) < 5.0 / math.sqrt(d) and abs(z[b].std() - 1.0) < 5.0 / math.sqrt(d)
    assert abs(np.corrcoef(z[0], z[1])[0, 1]) < 5.0 / math.sqrt(d)
    # counter-based: a value depends on (seed, row, coordinate) only
    short = oracle.attack("random", None, 2, 1.0, seed=12345, d=1001)
    assert np.array_equal(short, z[:2, :1001].astype(np.float32))
    other = oracle.attack("random", None, 1, 1.0, seed=12346, d=1001)
    assert not np.array_equal(other[0], short[0])
    scaled = oracle.attack("random", None, 1, -4.0, seed=12345, d=1001)
    assert np.array_equal(scaled[0], (np.float64(-4.0) * z[0, :1001]).astype(np.float32))


@pytest.mark.parametrize("ex", _golden()["attacks"], ids=lambda e: str(len(e["honest"])))
def test_attacks_hand_worked(ex):
    x = np.array(ex["honest"], dtype=np.float32)
    nb = ex["nbyz"]
    if "reverse" in ex:
        got = oracle.attack("reverse", x, nb, ex["reverse"]["param"])
        assert got.tolist() == ex["reverse"]["byz"]
    for kind in ("little", "empire"):
        got = oracle.attack(kind, x, nb, ex[kind]["param"])
        want = np.array(ex[kind]["byz_row"], dtype=np.float32)
        for b in range(nb):
            assert np.array_equal(got[b], want), (kind, got[b], want)


def test_moment_attacks_equal_numpy():
    rng = np.random.default_rng(21)
    for h in (1, 2, 5, 15, 64):
        x = (rng.standard_normal((h, 777)) * 0.01 + rng.standard_normal(777) * 0.01).astype(np.float32)
        xd = x.astype(np.float64)
        mean, std = xd.mean(axis=0), xd.std(axis=0, ddof=0)
        lie = oracle.attack("little", x, 4, 1.5)
        foe = oracle.attack("empire", x, 2, 0.1)
        want_lie = (mean - 1.5 * std).astype(np.float32)
        want_foe = (-0.1 * mean).astype(np.float32)
        # numpy's pairwise sums differ from the oracle's sequential ones in the
        # last fp64 bits only: at most one fp32 rounding step apart
        assert np.all(np.abs(lie - want_lie) <= np.spacing(np.abs(want_lie))), h
        assert np.all(np.abs(foe - want_foe) <= np.spacing(np.abs(want_foe))), h
        assert all(np.array_equal(lie[b], lie[0]) for b in range(4))
    # identical honest rows: the attack vector is that row (std 0)
    row = rng.standard_normal(50).astype(np.float32)
    assert np.array_equal(oracle.attack("little", np.tile(row, (7, 1)), 1, 3.0)[0], row)


def test_reverse_is_an_exact_scaling():
    rng = np.random.default_rng(22)
    x = rng.standard_normal((3, 101)).astype(np.float32)
    got = oracle.attack("reverse", x, 5, -100.0)
    for b in range(5):
        assert np.array_equal(got[b], (np.float64(-100.0) * x[b % 3].astype(np.float64)).astype(np.float32))
    assert np.array_equal(oracle.attack("reverse", x, 2, 0.5), x[:2] * np.float32(0.5))


@pytest.mark.parametrize("ex", _golden()["variance"], ids=lambda e: str(e["stats"]))
def test_variance_hand_worked(ex):
    s = oracle.variance_stats(np.array(ex["g"], np.float32), np.array(ex["grad"], np.float32))
    assert s.tolist() == ex["stats"]


def test_variance_equals_numpy_and_the_distance_identity():
    rng = np.random.default_rng(23)
    for h, d in [(2, 10), (9, 4097), (33, 1000), (64, 300)]:
        g = rng.standard_normal((h, d)).astype(np.float32)
        t = rng.standard_normal(d).astype(np.float32)
        s = oracle.variance_stats(g, t)
        want = np.var(g.astype(np.float64), axis=0, ddof=1).sum()
        assert s[0] == pytest.approx(want, rel=1e-12)
        D = oracle.pairwise_sqdist(g)
        assert s[0] == pytest.approx(np.triu(D, 1).sum() / (h * (h - 1)), rel=1e-12)
        assert s[1] == pytest.approx(float(np.dot(t.astype(np.float64), t.astype(np.float64))), rel=1e-12)


@pytest.mark.parametrize("ex", _golden()["delta"], ids=lambda e: f"n{e['n']}f{e['f']}")
def test_delta_closed_forms(ex):
    for rule, want in ex["values"].items():
        got = oracle.delta(rule, ex["n"], ex["f"])
        if want is None:
            assert math.isnan(got), rule
        else:
            assert got == pytest.approx(want, rel=1e-14), rule
    assert math.isnan(oracle.delta("bulyan", 11, 2))


def test_invalid_arguments():
    x = np.zeros((2, 3), np.float32)
    with pytest.raises(oracle.OracleError):
        oracle.variance_stats(x[:1], np.zeros(3, np.float32))   # h < 2
    with pytest.raises(KeyError):
        oracle.attack("drop", x, 1, 0.0)
