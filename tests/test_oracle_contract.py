"""Pins for the oracle's contraction step (no GPU): hand-worked steps
(tests/golden/contraction_examples.json), Average against the product with the
row-stochastic peer matrix (numpy), and the range invariants of Median and
Average (every output coordinate lies within its peers' values, so the spread
of the nodes' vectors cannot grow)."""
import json
import os
from fractions import Fraction

import numpy as np
import pytest

import oracle

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "contraction_examples.json")


def _golden():
    with open(GOLDEN) as fh:
        return json.load(fh)


@pytest.mark.parametrize("case", _golden()["cases"], ids=lambda c: c["name"])
def test_hand_worked_steps(case):
    x = np.array(_golden()["x"], dtype=np.float32)
    y, sel = oracle.contract_step(case["rule"], x, case["peers"], case["f"])
    want = np.array([[np.float32(float(Fraction(v))) for v in row] for row in case["y"]])
    assert np.array_equal(y, want)
    if "sel" in case:
        assert sel == case["sel"]


def _peers(n, q, rng):
    return np.stack([rng.permutation(n)[:q] for _ in range(n)]).astype(np.int32)


def test_average_is_the_peer_matrix_product():
    rng = np.random.default_rng(4)
    n, q, d = 12, 7, 513
    x = rng.standard_normal((n, d)).astype(np.float32)
    peers = _peers(n, q, rng)
    P = np.zeros((n, n))
    for v in range(n):
        P[v, peers[v]] = 1.0 / q
    y, _ = oracle.contract_step("average", x, peers, 0)
    want = (P @ x.astype(np.float64)).astype(np.float32)
    assert np.all(np.abs(y - want) <= np.spacing(np.abs(want)))


@pytest.mark.parametrize("rule,q,f", [("median", 7, 3), ("average", 5, 0), ("median", 8, 2)])
def test_outputs_stay_within_the_peers_range(rule, q, f):
    rng = np.random.default_rng(q + f)
    n, d = 10, 301
    x = rng.standard_normal((n, d)).astype(np.float32)
    peers = _peers(n, q, rng)
    y, _ = oracle.contract_step(rule, x, peers, f)
    for v in range(n):
        lo, hi = x[peers[v]].min(0), x[peers[v]].max(0)
        assert np.all(y[v] >= lo) and np.all(y[v] <= hi)
        if rule == "median" and q % 2 == 1:
            assert np.all((x[peers[v]] == y[v]).any(0))  # an input value, bit for bit
    spread = lambda a: (a.max(0) - a.min(0)).max()
    assert spread(y) <= spread(x)


def test_all_peers_in_order_reduce_to_the_rule():
    rng = np.random.default_rng(8)
    n, d, f = 11, 257, 2
    x = rng.standard_normal((n, d)).astype(np.float32)
    peers = np.tile(np.arange(n, dtype=np.int32), (n, 1))
    for rule, fn in (("multikrum", lambda: oracle.multikrum(x, f)),
                     ("mda", lambda: oracle.mda(x, f)),
                     ("bulyan", lambda: oracle.bulyan(np.ascontiguousarray(x[:9]), 1))):
        if rule == "bulyan":
            y, sel = oracle.contract_step(rule, x[:9], peers[:9, :9], 1)
        else:
            y, sel = oracle.contract_step(rule, x, peers, f)
        out, s = fn()[:2]
        assert all(np.array_equal(row, out) for row in y) and all(t == s.tolist() for t in sel)
