"""GPU parity of contraction steps (every node aggregating its peers at once).

Nodes hear random peer lists (some including themselves, in random order).
For each node whose decisions are all pinned (the pinning checks of
tests/parity.py on the node's own sub-matrix of distances and bounds), the
selected rows must equal the oracle's; every output row must match the
oracle's within max(1e-5 |oracle|, 1e-6) (Krum, Median and Average bit for
bit: a copy, an input value, and the same fp64 sum in the same order). With
every node hearing all n nodes in order, each row equals the plain rule call
bit for bit. Both distance engines are covered (n <= 20 direct, larger Gram).
"""
import numpy as np
import pytest
import torch

import oracle
import parity
import paper_2010_05888_amd as gf

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


@pytest.fixture(scope="module", autouse=True)
def _library():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    gf.load()
    gf.set_direct_max_n(20)


def _inputs(n, d, seed):
    rng = np.random.default_rng(seed)
    x = (rng.standard_normal((n, d)) * (1.0 + rng.permutation(n)[:, None] / n)).astype(np.float32)
    x[: max(1, n // 8)] *= 10.0
    return rng, x


def _pinned_nodes(rule, x, peers, f, m, B):
    ok = []
    D = oracle.pairwise_sqdist(x)
    for v in range(x.shape[0]):
        p = list(peers[v])
        xs = np.ascontiguousarray(x[p])
        Ds, Bs = D[np.ix_(p, p)], B[np.ix_(p, p)]
        same = parity.identical_rows(Ds)
        if rule in ("krum", "multikrum"):
            mm = 1 if rule == "krum" else m
            _, _, sc = oracle.multikrum(xs, f, mm, return_scores=True)
            ok.append(parity.krum_pinned(sc, Ds, Bs, f, mm, same)[0])
        elif rule in ("bulyan", "multikrum_iterated"):
            res = (oracle.bulyan(xs, f, return_rounds=True) if rule == "bulyan"
                   else oracle.multikrum_iterated(xs, f, m, return_rounds=True))
            ok.append(parity.bulyan_pinned(res[2], res[3], Ds, Bs, len(p), f, same)[0])
        elif rule == "mda":
            _, sel = oracle.mda(xs, f)
            ok.append(parity.mda_pinned(Ds, Bs, len(p), f, sel)[0])
        else:
            ok.append(True)
    return ok


CASES = [("average", 0, None), ("median", 3, None), ("krum", 2, None), ("multikrum", 2, 5),
         ("multikrum_iterated", 2, 5), ("bulyan", 2, None), ("mda", 2, None)]


@pytest.mark.parametrize("n,q,d", [(12, 11, 5003), (20, 15, 4097), (40, 23, 3001)])
@pytest.mark.parametrize("rule,f,m", CASES)
def test_step_matches_the_oracle(rule, f, m, n, q, d):
    rng, x = _inputs(n, d, 1000 * n + q)
    peers = np.stack([rng.permutation(n)[:q] for _ in range(n)]).astype(np.int32)
    xt = torch.from_numpy(x).to(DEV)
    pt = torch.from_numpy(peers).to(DEV)
    y = gf.contract_step(rule, xt, pt, f, m).cpu().numpy()
    want, want_sel = oracle.contract_step(rule, x, peers, f, m)
    eng = gf.distance_engine(n, d)
    ref = parity.checked_reference(x, gf.gram_reference(xt)) if eng == "gram" else None
    B = parity.dist_bounds(oracle.pairwise_sqdist(x), eng, ref, x)
    pinned = _pinned_nodes(rule, x, peers, f, m, B)
    assert sum(pinned) >= n // 2, "too few pinned nodes to test"
    for v in range(n):
        if not pinned[v]:
            continue
        if rule in ("krum", "median", "average"):
            assert np.array_equal(y[v], want[v]), (rule, v)
        else:
            ok, at, err = parity.agg_close(y[v], want[v])
            assert ok, (rule, v, at, err)


@pytest.mark.parametrize("rule,f", [("multikrum", 2), ("bulyan", 2), ("median", 3), ("krum", 1),
                                    ("multikrum_iterated", 2), ("average", 0), ("mda", 2)])
@pytest.mark.parametrize("n", [11, 33])
def test_all_peers_in_order_equal_the_plain_rule(rule, f, n):
    if rule == "bulyan" and n < 4 * f + 3:
        pytest.skip("below Bulyan's requirement")
    _, x = _inputs(n, 7001, n)
    xt = torch.from_numpy(x).to(DEV)
    peers = torch.arange(n, dtype=torch.int32, device=DEV).repeat(n, 1)
    y = gf.contract_step(rule, xt, peers, f)
    if rule == "average":
        want = gf.average(xt)
    else:
        want = gf.gar(rule, xt, f)[0]
    assert all(torch.equal(y[v], want) for v in range(n))


def test_mda_with_64_peers():
    # 64 peers per node: the subset search's dynamic LDS (D, prefix maxima and
    # indices) exceeds 64 KB and is requested from the runtime
    n, f = 64, 2
    _, x = _inputs(n, 3001, 64)
    xt = torch.from_numpy(x).to(DEV)
    peers = torch.arange(n, dtype=torch.int32, device=DEV).repeat(n, 1)
    y = gf.contract_step("mda", xt, peers, f)
    want = gf.gar("mda", xt, f)[0]
    assert all(torch.equal(y[v], want) for v in range(n))


def test_several_steps():
    n, q, d, f = 16, 9, 2049, 2
    rng, x = _inputs(n, d, 5)
    peers = np.stack([rng.permutation(n)[:q] for _ in range(n)]).astype(np.int32)
    xt = torch.from_numpy(x).to(DEV)
    pt = torch.from_numpy(peers).to(DEV)
    got = gf.contract("median", xt, pt, f, 3).cpu().numpy()
    want = x
    for _ in range(3):
        want, _ = oracle.contract_step("median", want, peers, f)
    assert np.array_equal(got, want)
    spread = lambda a: (a.max(0) - a.min(0)).max()
    assert spread(got) <= spread(x)


def test_invalid_arguments_are_rejected():
    x = torch.zeros((6, 10), dtype=torch.float32, device=DEV)
    p = torch.zeros((6, 7), dtype=torch.int32, device=DEV)
    with pytest.raises(gf.GarfieldError) as e:
        gf.contract_step("median", x, p, 0)  # q > n
    assert e.value.code == gf.EINVAL
    p = torch.arange(5, dtype=torch.int32, device=DEV).repeat(6, 1)
    with pytest.raises(gf.GarfieldError) as e:
        gf.contract_step("dist", x, p, 1)
    assert e.value.code == gf.EINVAL
    with pytest.raises(gf.GarfieldError) as e:
        gf.contract_step("krum", x, p, 2)  # q = 5 < 2f+3
    assert e.value.code == gf.EREQ
    x = torch.zeros((30, 10), dtype=torch.float32, device=DEV)
    p = torch.arange(30, dtype=torch.int32, device=DEV).repeat(30, 1)
    with pytest.raises(gf.GarfieldError) as e:
        gf.contract_step("mda", x, p, 8)  # C(30, 8) subsets per node, above the per-node cap
    assert e.value.code == gf.ETOOBIG


def test_mda_small_integer_ties():
    # exact distances: many equal diameters, the first subset of positions wins
    rng = np.random.default_rng(9)
    for trial in range(10):
        n = int(rng.integers(5, 16))
        q = int(rng.integers(3, n + 1))
        f = int(rng.integers(0, (q - 1) // 2 + 1))
        x = rng.integers(-2, 3, size=(n, 33)).astype(np.float32)
        peers = np.stack([rng.permutation(n)[:q] for _ in range(n)]).astype(np.int32)
        y = gf.contract_step("mda", torch.from_numpy(x).to(DEV), torch.from_numpy(peers).to(DEV), f)
        want, want_sel = oracle.contract_step("mda", x, peers, f)
        got = y.cpu().numpy()
        for v in range(n):  # exact sums of small integers: equal iff the same rows were taken
            assert np.array_equal(got[v], want[v]), (trial, n, q, f, v, want_sel[v])
