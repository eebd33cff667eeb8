"""GPU invariants of every rule, checked without the oracle.

Each rule is a function of the set of n vectors (Section 3.1), so on the
library's own outputs:

* permuting the rows permutes the selection and leaves the aggregate as it
  was: bit for bit for Krum (a copy), the median (an order statistic) and
  Bulyan (its beta values are summed in the order of their distance to the
  median, not of their row index); within the aggregate tolerance for the
  means of Multi-Krum, MDA and Average, which add the rows in index order;
* scaling by 2^s leaves every selection as it was and scales every aggregate
  by 2^s exactly (every fp operation of the direct engine scales exactly, and
  the Gram engine's per-row quantization exponent moves by s);
* negating the rows leaves the selections as they were and negates the
  aggregates (Bulyan's within tolerance: its tie rule between values equally
  far from the median prefers the smaller one).

Both distance engines run at n = 11; n = 33 takes the Gram engine and MDA's
vertex-cover search (C(33, 7) subsets).
"""
import numpy as np
import pytest
import torch

import parity
import paper_2010_05888_amd as gf

pytestmark = pytest.mark.gpu
DEV = "cuda:0"

RULES = ["krum", "multikrum", "median", "bulyan", "mda", "average"]
PERMUTATION_EXACT = {"krum", "median", "bulyan"}
CASES = [(11, 2, "direct"), (11, 2, "gram"), (33, 7, "gram")]


@pytest.fixture(scope="module", autouse=True)
def _library():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    gf.load()  # raises if libgarfield.so is missing: no fallback exists
    yield
    gf.set_direct_max_n(20)


def _data(n, f, seed):
    # distinct row scales and f far rows: well-separated scores, no ties
    rng = np.random.default_rng(seed)
    d = 20011
    x = (rng.standard_normal((n, d)) * (1.0 + 0.5 * rng.permutation(n)[:, None] / n)).astype(np.float32)
    x[:f] *= 8.0
    return x, rng


def _run(rule, x, f):
    out, sel = gf.gar(rule, x, f)
    torch.cuda.synchronize()
    return out, (None if sel is None else sel.cpu().numpy())


@pytest.mark.parametrize("n,f,engine", CASES)
@pytest.mark.parametrize("rule", RULES)
def test_permutation_scaling_negation(rule, n, f, engine):
    old = gf.set_direct_max_n(20 if engine == "direct" else 1)
    try:
        x, rng = _data(n, f, 7000 + 10 * n + RULES.index(rule))
        xt = torch.from_numpy(x).to(DEV)
        out, sel = _run(rule, xt, f)

        perm = rng.permutation(n)
        outp, selp = _run(rule, torch.from_numpy(x[perm]).to(DEV), f)
        if sel is not None:
            assert sorted(perm[selp].tolist()) == sel.tolist(), "permutation moved the selection"
        if rule in PERMUTATION_EXACT:
            assert torch.equal(outp, out)
        else:
            ok, at, err = parity.agg_close(outp.cpu().numpy(), out.cpu().numpy())
            assert ok, (at, err)

        for s in (-3, 5):
            outs, sels = _run(rule, xt * float(2.0 ** s), f)
            if sel is not None:
                assert sels.tolist() == sel.tolist(), f"scaling by 2^{s} moved the selection"
            assert torch.equal(outs, out * float(2.0 ** s)), f"scaling by 2^{s}"

        outn, seln = _run(rule, -xt, f)
        if sel is not None:
            assert seln.tolist() == sel.tolist(), "negation moved the selection"
        if rule == "bulyan":
            ok, at, err = parity.agg_close(outn.cpu().numpy(), (-out).cpu().numpy())
            assert ok, (at, err)
        else:
            assert torch.equal(outn, -out)
    finally:
        gf.set_direct_max_n(old)


@pytest.mark.parametrize("n,f,engine", CASES + [(64, 15, "gram")])
def test_distance_matrix_permutes_and_scales_exactly(n, f, engine):
    # D of the permuted rows is D permuted, bit for bit (each entry depends on
    # its two rows only: per pair in the direct engine; through exact integer
    # products of rows shifted by the same reference row in the Gram engine),
    # and D of 2^s x is 4^s D exactly
    old = gf.set_direct_max_n(20 if engine == "direct" else 1)
    try:
        x, rng = _data(n, f, 9100 + n)
        xt = torch.from_numpy(x).to(DEV)
        D = gf.pairwise_sqdist(xt).cpu().numpy()
        perm = rng.permutation(n)
        Dp = gf.pairwise_sqdist(torch.from_numpy(x[perm]).to(DEV)).cpu().numpy()
        assert np.array_equal(Dp, D[np.ix_(perm, perm)])
        for s in (-3, 5):
            Ds = gf.pairwise_sqdist(xt * float(2.0 ** s)).cpu().numpy()
            assert np.array_equal(Ds, D * 4.0 ** s), f"scaling by 2^{s}"
        assert np.array_equal(gf.pairwise_sqdist(-xt).cpu().numpy(), D)
    finally:
        gf.set_direct_max_n(old)
