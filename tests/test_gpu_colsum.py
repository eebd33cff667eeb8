"""The mean of a large Multi-Krum selection from the distance pass's column sums.

For n <= 12 and 2m > n + 4 the distance pass also stores every coordinate's
fp64 sum over all n rows, or NaN where the exponents of the coordinate's
values span more than 23 binades (then a sum of some of the rows might not be
exact), and the mean subtracts the unselected rows from it. Where it is exact
this is the same fp64 value as the selected rows' sum in ascending order, so
the aggregate must equal the oracle's bit for bit on both paths: ordinary
values, and coordinates with huge, tiny, subnormal and zero values mixed.
"""
import numpy as np
import pytest
import torch

import oracle
import paper_2010_05888_amd as gf

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _rows(n, d, seed):
    """Small-integer rows (exact distances, so the selection is decided
    exactly) whose first two rows are far from the rest."""
    rng = np.random.default_rng(seed)
    x = rng.integers(-3, 4, size=(n, d)).astype(np.float32)
    x[:2] += 40.0
    return x, rng


def _check(x, f, m, rule="multikrum"):
    xt = torch.from_numpy(x).to(DEV)
    if rule == "multikrum":
        out, sel = gf.multikrum(xt, f, m)
        oo, so = oracle.multikrum(x, f, m)
    elif rule == "mda":
        out, sel = gf.mda(xt, f)
        oo, so = oracle.mda(x, f)
    else:
        out, sel = gf.multikrum_iterated(xt, f, m)
        oo, so = oracle.multikrum_iterated(x, f, m)
    torch.cuda.synchronize()
    assert sel.cpu().numpy().tolist() == so.tolist()
    got = out.cpu().numpy()
    bad = np.flatnonzero(got.view(np.uint32) != oo.view(np.uint32))
    assert bad.size == 0, (bad[:5], got[bad[:5]], oo[bad[:5]])


@pytest.mark.parametrize("n,f,m,d", [(11, 2, 9, 50003), (12, 2, 10, 4097), (7, 1, 6, 1),
                                     (7, 1, 6, 4099)])
def test_exact_path_matches_the_oracle(n, f, m, d):
    assert 2 * m > n + 4
    x, rng = _rows(n, d, n * 1000 + d)
    x += rng.standard_normal((n, d)).astype(np.float32) * 0.25
    print(f"colsum exact n={n} m={m} d={d}", flush=True)
    _check(x, f, m)


@pytest.mark.parametrize("rule", ["multikrum", "multikrum_iterated", "mda"])
def test_inexact_coordinates_take_the_row_sum(rule):
    n, f, m, d = 11, 2, 9, 20011
    x, rng = _rows(n, d, 77)
    cols = rng.permutation(d)
    huge, tiny, sub, zero, mixed = np.array_split(cols[:5000], 5)
    x[0, huge] = 3.0e17           # an excluded row far beyond the others: not exact
    x[1, huge] = -2.5e17
    x[5, tiny] = 1.0e-20          # a selected row below the others: not exact
    x[:, sub] = 0.0
    x[3, sub] = 1.0e-40           # a subnormal among zeros: exact
    x[4, sub] = -3.0e-41
    x[:, zero] = 0.0
    x[6, zero] = -0.0             # all zeros: exact, +0
    x[7, mixed] = 2.0 ** 23       # 23 binades above 1: still exact
    x[8, mixed] = 1.0
    print(f"colsum inexact {rule}", flush=True)
    _check(x, f, m, rule)


def test_workspace_includes_the_column_sums():
    d = 1 << 20
    with_sums = gf.workspace_bytes("multikrum", 11, 2, d, 9)
    without = gf.workspace_bytes("multikrum", 11, 2, d, 7)  # 2m <= n + 4
    assert with_sums - without >= 8 * d


@pytest.mark.parametrize("d", [4099, 4100])
def test_rows_at_an_odd_float_offset(d):
    # rows starting one float past 16-byte alignment: both kernels still load
    # 16 bytes per lane, from addresses that are only float-aligned (f4u)
    n, f, m = 11, 2, 9
    x, rng = _rows(n, d, 5 + d)
    x += rng.standard_normal((n, d)).astype(np.float32)
    x[0, ::7] = 1.0e20
    buf = torch.empty(n * d + 1, dtype=torch.float32, device=DEV)
    xt = buf[1:].view(n, d)
    xt.copy_(torch.from_numpy(x))
    out, sel = gf.multikrum(xt, f, m)
    oo, so = oracle.multikrum(x, f, m)
    torch.cuda.synchronize()
    assert sel.cpu().numpy().tolist() == so.tolist()
    assert np.array_equal(out.cpu().numpy().view(np.uint32), oo.view(np.uint32))
