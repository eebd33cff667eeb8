"""MDA's search through vertex covers (Section 3.1 item 3), used from 2^20
candidate subsets C(n, f) on: the least diameter is the smallest pair distance
whose graph of farther pairs has a vertex cover of at most f vectors (a binary
search over the sorted distances, each step a bounded search-tree test), and
the winner, the lexicographically first subset of that diameter, is built
vertex by vertex with the same test.

Checked bit for bit against the oracle's enumeration (integer rows give exact
distances on both sides, so diameters tie and the first subset in
lexicographic order must win), and against the library's own enumeration of
every subset at sizes the oracle cannot enumerate in seconds (both read the
same device distances, so they must pick the same subset).
"""
from math import comb

import numpy as np
import pytest
import torch

import oracle
import paper_2010_05888_amd as gf

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
ENUMERATE = 1 << 62  # threshold above any C(n, f) the library accepts: always enumerate


@pytest.fixture(scope="module", autouse=True)
def _library():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    gf.load()
    yield


@pytest.fixture
def cover():
    old = gf.set_mda_cover_min(0)  # every MDA call searches by covers
    yield
    gf.set_mda_cover_min(old)


def _to_dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


def _both(xt, f):
    """(cover, enumeration) results of garfield_mda on the same input."""
    old = gf.set_mda_cover_min(0)
    try:
        a = gf.mda(xt, f)
        gf.set_mda_cover_min(ENUMERATE)
        b = gf.mda(xt, f)
    finally:
        gf.set_mda_cover_min(old)
    return a, b


def test_small_integer_ties_against_oracle(cover):
    rng = np.random.default_rng(21)
    for trial in range(60):
        n = int(rng.integers(1, 17))
        d = int(rng.choice([1, 2, 5, 33]))
        lim = int(rng.choice([1, 2, 40]))
        x = rng.integers(-lim, lim + 1, size=(n, d)).astype(np.float32)
        xt = _to_dev(x)
        for f in sorted({0, (n - 1) // 2, max(0, (n - 1) // 4)}):
            out, sel = gf.mda(xt, f)
            oo, so = oracle.mda(x, f)
            assert sel.cpu().tolist() == so.tolist(), (trial, n, d, lim, f)
            assert np.array_equal(out.cpu().numpy(), oo), (trial, n, d, lim, f)


def test_degenerate_inputs(cover):
    # identical rows: every diameter is 0, so the first n - f rows win
    x = np.ones((9, 50), dtype=np.float32)
    _, sel = gf.mda(_to_dev(x), 4)
    assert sel.cpu().tolist() == [0, 1, 2, 3, 4]
    # one row, f = 0; two clusters where dropping one cluster is the only cover
    _, sel = gf.mda(_to_dev(np.zeros((1, 3), np.float32)), 0)
    assert sel.cpu().tolist() == [0]
    x = np.zeros((11, 4), dtype=np.float32)
    x[[1, 4, 6]] = 100.0
    _, sel = gf.mda(_to_dev(x), 3)
    assert sel.cpu().tolist() == [0, 2, 3, 5, 7, 8, 9, 10]
    # zero dimension: all distances 0
    _, sel = gf.mda(torch.empty((7, 0), device=DEV), 3)
    assert sel.cpu().tolist() == [0, 1, 2, 3]


@pytest.mark.parametrize("n,f,d,lim", [(27, 6, 33, 2), (31, 7, 33, 2), (34, 7, 3, 20),
                                       (40, 6, 2, 50), (33, 16, 4, 3)])
def test_many_subsets(n, f, d, lim):
    # integer rows: ties in 33 dimensions of [-2, 2], spread distances in 2 or 3
    # dimensions of a wide range; the oracle enumerates up to a few million
    rng = np.random.default_rng(n * 7 + f + d)
    x = rng.integers(-lim, lim + 1, size=(n, d)).astype(np.float32)
    (oa, sa), (ob, sb) = _both(_to_dev(x), f)
    assert torch.equal(sa, sb) and torch.equal(oa, ob), (sa.tolist(), sb.tolist())
    if comb(n, f) <= 6_000_000:
        oo, so = oracle.mda(x, f)
        assert sa.cpu().tolist() == so.tolist()
        assert np.array_equal(oa.cpu().numpy(), oo)


@pytest.mark.parametrize("n,f,d", [(12, 3, 1000), (19, 4, 4097), (25, 8, 2000), (31, 7, 20011),
                                   (39, 9, 100000), (64, 7, 3000), (64, 1, 50)])
def test_cover_equals_enumeration(n, f, d):
    # Gaussian rows: distinct diameters, the Gram engine above n = 20
    g = torch.Generator(device=DEV).manual_seed(n * 1000 + f)
    xt = torch.randn((n, d), device=DEV, generator=g)
    xt[: f // 2] *= 1.5
    (oa, sa), (ob, sb) = _both(xt, f)
    assert torch.equal(sa, sb), (sa.tolist(), sb.tolist())
    assert torch.equal(oa, ob)


def test_fig3_shape_n39():
    # the micro-benchmark's n = 39, f = 9 (211 million subsets) at d = 10^7
    g = torch.Generator(device=DEV).manual_seed(39)
    xt = torch.randn((39, 10_000_000), device=DEV, generator=g)
    (oa, sa), (ob, sb) = _both(xt, 9)
    assert torch.equal(sa, sb)
    assert torch.equal(oa, ob)
