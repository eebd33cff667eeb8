"""The Gram engine's reference-row rule as the tests evaluate it (parity.py),
pinned on hand-worked inputs and by brute force, so that the GPU tests check
the library's pick against something other than the library."""
from itertools import combinations

import numpy as np

import parity


def test_hand_worked_rows():
    # d = 1, rows 0, 1, 2, 100, 3; n = 5, so each score is the sum of the 3
    # smallest squared distances, self included: row 0: 0 + 1 + 4 = 5,
    # row 1: 0 + 1 + 1 = 2, row 2: 0 + 1 + 1 = 2, row 3: 0 + 9409 + 9604,
    # row 4: 0 + 1 + 4 = 5. Rows 1 and 2 tie; the lower index wins.
    x = np.array([[0.0], [1.0], [2.0], [100.0], [3.0]], dtype=np.float32)
    best, cands = parity.gram_reference_rule(x)
    assert best == 1
    assert cands == [1, 2]  # an exact tie in exact arithmetic is not separable


def test_identical_rows_tie_to_the_lower_index():
    # three copies of the central row: the copies with higher indices are not
    # candidates (the library's probe rows are bit-identical, so it breaks the
    # tie by index as the rule does)
    rng = np.random.default_rng(1)
    x = rng.standard_normal((9, 40)).astype(np.float32)
    x[[2, 5, 7]] = 0.0
    best, cands = parity.gram_reference_rule(x)
    assert best == 2 and 5 not in cands and 7 not in cands


def test_sample_of_long_rows():
    # d > 1024: only 4 runs of 256 coordinates at r * (d // 4) count; a row that
    # is central on the sample wins even if it is far away elsewhere
    d = 10_000
    rng = np.random.default_rng(2)
    x = (rng.standard_normal((7, d)) * 0.1).astype(np.float32)
    x[4] = 0.0
    cols = np.concatenate(parity.probe_columns(d))
    assert cols.size == 1024 and cols[0] == 0 and cols[256] == d // 4
    off = np.setdiff1d(np.arange(d), cols)
    x[4, off] = 50.0
    best, _ = parity.gram_reference_rule(x)
    assert best == 4


def test_against_brute_force():
    # the score as a minimum over subsets: the least sum of distances to any
    # ceil(n/2) rows (self included) equals the sum of the ceil(n/2) smallest
    rng = np.random.default_rng(3)
    for trial in range(40):
        n = int(rng.integers(2, 9))
        d = int(rng.integers(1, 6))
        x = rng.integers(-4, 5, size=(n, d)).astype(np.float32)
        h = (n + 1) // 2
        P = ((x[:, None, :].astype(np.int64) - x[None, :, :]) ** 2).sum(-1)
        score = [min(sum(P[i, j] for j in S) for S in combinations(range(n), h) if i in S)
                 for i in range(n)]
        want = min(range(n), key=lambda i: (score[i], i))
        best, cands = parity.gram_reference_rule(x)
        assert best == want, (trial, x.tolist())
        assert want in cands
