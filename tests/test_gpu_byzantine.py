"""GPU parity of the Byzantine vectors and the variance condition.

Every attack kind and the variance statistics run through the C-ABI and are
compared with the CPU oracle on the same seeded inputs, at dimensions with a
ragged tail, on misaligned rows (a view one float into an allocation), and at
the edges (d = 0, nbyz = 0, h = 1, nbyz = 64). Tolerances:

* reversed vectors: bit-exact (one fp64 product rounded once on both sides);
* fall of empires: at most one fp32 rounding step (both sides form the mean in
  fp64, in different orders);
* little is enough: one fp32 rounding step plus the fp64 error of the two
  moment computations, far below it;
* random vectors: |sigma| * 3e-6 absolute. The kernel evaluates Box-Muller in
  fp32 (log, sincospi and sqrt, each within about an ulp), the oracle in fp64,
  from the same Philox words and the same exact uniforms; r = sqrt(-2 ln u)
  is at most 5.8, so the fp32 error is below 5.8 * 2^-21 sigma;
* variance estimate: the sum over pairs of the distance engine's error bound
  (tests/parity.py) divided by h (h - 1); ||grad||^2 within 4 d 2^-53
  relative (fp64 sums of exact squares in two orders).
"""
import math

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
    yield
    gf.set_direct_max_n(20)


def _dev(x, misalign=False):
    x = np.ascontiguousarray(x, dtype=np.float32)
    if not misalign:
        return torch.from_numpy(x).to(DEV)
    flat = torch.empty(x.size + 1, dtype=torch.float32, device=DEV)
    view = flat[1:].view(x.shape)
    view.copy_(torch.from_numpy(x))
    return view


def _out(nbyz, d, misalign=False):
    flat = torch.full((nbyz * d + 1,), float("nan"), dtype=torch.float32, device=DEV)
    return (flat[1:] if misalign else flat[:-1]).view(nbyz, d), flat


def _honest(h, d, seed):
    rng = np.random.default_rng(seed)
    mu = rng.standard_normal(d) * 0.01
    return (mu + rng.standard_normal((h, d)) * 0.01).astype(np.float32)


SHAPES = [(1, 1, 1), (2, 3, 5), (15, 4, 4097), (9, 2, 10003), (64, 64, 1031), (5, 1, 65536)]


@pytest.mark.parametrize("misalign", [False, True])
@pytest.mark.parametrize("h,nbyz,d", SHAPES)
def test_reverse_is_bit_exact(h, nbyz, d, misalign):
    x = _honest(h, d, 1 + h + d)
    out, _ = _out(nbyz, d, misalign)
    gf.attack("reverse", _dev(x, misalign), nbyz, -100.0, out=out)
    assert np.array_equal(out.cpu().numpy(), oracle.attack("reverse", x, nbyz, -100.0))


@pytest.mark.parametrize("misalign", [False, True])
@pytest.mark.parametrize("h,nbyz,d", SHAPES)
def test_moment_attacks(h, nbyz, d, misalign):
    x = _honest(h, d, 2 + h + d)
    xd = x.astype(np.float64)
    scale = np.abs(xd.mean(0)) + 1.5 * xd.std(0)
    for kind, param in (("little", 1.5), ("empire", 0.1), ("little", -3.0)):
        out, _ = _out(nbyz, d, misalign)
        gf.attack(kind, _dev(x, misalign), nbyz, param, out=out)
        got = out.cpu().numpy()
        want = oracle.attack(kind, x, nbyz, param)
        tol = np.spacing(np.abs(want).astype(np.float32)) + 1e-12 * scale * max(1.0, abs(param))
        assert np.all(np.abs(got.astype(np.float64) - want) <= tol), (kind, param)
        assert all(np.array_equal(got[b], got[0]) for b in range(nbyz))


@pytest.mark.parametrize("misalign", [False, True])
@pytest.mark.parametrize("nbyz,d", [(1, 1), (2, 3), (4, 4097), (64, 1031), (3, 100003)])
def test_random_matches_the_oracle(nbyz, d, misalign):
    for sigma, seed in ((1.0, 0), (0.01, 2010058882), (-7.5, 2**63 + 5)):
        out, _ = _out(nbyz, d, misalign)
        gf.attack("random", None, nbyz, sigma, seed=seed, out=out)
        got = out.cpu().numpy().astype(np.float64)
        want = oracle.attack("random", None, nbyz, sigma, seed=seed, d=d).astype(np.float64)
        err = np.abs(got - want).max()
        assert err <= abs(sigma) * 3e-6, (sigma, seed, err)


def test_random_rows_do_not_depend_on_the_launch():
    # the same seed gives the same prefix at any d and through any row window
    full, _ = _out(5, 9001)
    gf.attack("random", None, 5, 1.0, seed=77, out=full)
    short, _ = _out(2, 4000)
    gf.attack("random", None, 2, 1.0, seed=77, out=short)
    assert torch.equal(full[:2, :4000], short)


def test_attacks_write_only_their_rows():
    h, nbyz, d = 7, 3, 1025
    x = _honest(h, d, 5)
    out, flat = _out(nbyz, d)
    gf.attack("little", _dev(x), nbyz, 1.0, out=out)
    assert math.isnan(flat[-1].item())  # the float after the last row is untouched
    empty, _ = _out(0, d)
    assert gf.attack("empire", _dev(x), 0, 1.0, out=empty).numel() == 0
    z = torch.empty((3, 0), dtype=torch.float32, device=DEV)
    assert gf.attack("little", z, 2, 1.0).shape == (2, 0)


def test_attack_rows_feed_a_rule():
    # honest rows and Byzantine rows of one rule input, built in place
    h, f, d = 15, 4, 20011
    x = torch.empty((h + f, d), dtype=torch.float32, device=DEV)
    x[:h] = _dev(_honest(h, d, 9))
    gf.attack("little", x[:h], f, 1.5, out=x[h:])
    xn = x.cpu().numpy()
    assert np.array_equal(xn[h:], np.tile(xn[h], (f, 1)))
    oo, so, picks, rs = oracle.bulyan(xn, f, return_rounds=True)
    Do = oracle.pairwise_sqdist(xn)
    B = parity.dist_bounds(Do, gf.distance_engine(h + f, d))
    # this seeded input is pinned: the decisions are checked, never skipped
    assert parity.bulyan_pinned(picks, rs, Do, B, h + f, f, parity.identical_rows(Do))[0]
    out, sel = gf.bulyan(x, f)
    assert sel.cpu().numpy().tolist() == so.tolist()
    ok, at, err = parity.agg_close(out.cpu().numpy(), oo)
    assert ok, (at, err)


@pytest.mark.parametrize("engine", ["direct", "gram"])
@pytest.mark.parametrize("h,d", [(2, 1), (3, 7), (9, 11173), (11, 4099), (33, 20011), (64, 3001)])
def test_variance_stats(engine, h, d):
    old = gf.set_direct_max_n(20 if engine == "direct" else 1)
    try:
        g = _honest(h, d, 100 + h)
        t = np.random.default_rng(h).standard_normal(d).astype(np.float32)
        gt = _dev(g)
        got = gf.variance_stats(gt, _dev(t)).cpu().numpy()
        want = oracle.variance_stats(g, t)
        D = oracle.pairwise_sqdist(g)
        eng = gf.distance_engine(h, d)
        ref = parity.checked_reference(g, gf.gram_reference(gt)) if eng == "gram" else None
        B = parity.dist_bounds(D, eng, ref, g)
        tol0 = np.triu(B, 1).sum() / (h * (h - 1)) + 1e-12 * want[0]
        assert abs(got[0] - want[0]) <= tol0, (got[0], want[0], tol0)
        assert abs(got[1] - want[1]) <= 4 * d * 2.0 ** -53 * want[1]
    finally:
        gf.set_direct_max_n(old)


def test_variance_condition_and_delta():
    h, d = 9, 50001
    g = _honest(h, d, 31)
    grad = g.astype(np.float64).mean(0).astype(np.float32) * 40.0
    res = gf.variance_condition(_dev(g), _dev(grad), 11, 2)
    s = oracle.variance_stats(g, grad)
    for rule in ("mda", "krum", "median"):
        assert res[rule]["delta"] == pytest.approx(oracle.delta(rule, 11, 2), rel=1e-15)
        want = math.sqrt(s[1]) / (oracle.delta(rule, 11, 2) * math.sqrt(s[0]))
        assert res[rule]["ratio"] == pytest.approx(want, rel=1e-5)
        assert res[rule]["holds"] == (want > 1.0)
    assert math.isnan(gf.delta("bulyan", 11, 2)) and math.isnan(gf.delta("krum", 6, 2))


def test_variance_zero_dimension_and_identical_rows():
    z = torch.empty((4, 0), dtype=torch.float32, device=DEV)
    assert gf.variance_stats(z, torch.empty(0, device=DEV)).cpu().tolist() == [0.0, 0.0]
    row = np.random.default_rng(3).standard_normal(777).astype(np.float32)
    g = _dev(np.tile(row, (5, 1)))
    s = gf.variance_stats(g, g[0]).cpu().numpy()
    assert s[0] == 0.0 and s[1] == pytest.approx(float(np.dot(row.astype(np.float64), row)), rel=1e-12)


def test_invalid_arguments_are_rejected():
    x = torch.zeros((3, 10), dtype=torch.float32, device=DEV)
    out = torch.zeros((2, 10), dtype=torch.float32, device=DEV)
    for call, code in [
        (lambda: gf.attack("little", x, 65, 1.0), gf.ETOOBIG),
        (lambda: gf.attack("reverse", x, 2, float("nan"), out=out), gf.EINVAL),
        (lambda: gf.variance_stats(x[:1], x[0]), gf.EINVAL),
    ]:
        with pytest.raises(gf.GarfieldError) as e:
            call()
        assert e.value.code == code
