"""Krum / Multi-Krum of short inputs (n <= 12 rows, up to about 10^5
coordinates) in two launches: the distance pass, then one kernel whose
workgroups each add the distance partials, select, and write the mean of their
1,024 coordinates. It must make the same selection and write the same bits as
the separate selection and mean kernels (the tuning switch turns the combined
kernel off), and match the oracle: selection bit-exact, Krum's output a
bit-identical copy of the selected input, Multi-Krum's mean within the
aggregate tolerance.
"""
import numpy as np
import pytest
import torch

import oracle
import parity
import paper_2010_05888_amd as gf
from paper_2010_05888_amd import synth

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


@pytest.fixture(scope="module", autouse=True)
def _library():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    gf.load()
    yield
    gf.set_fused(True)


def _to_dev(x):
    return torch.from_numpy(np.ascontiguousarray(x)).to(DEV)


def _both(xt, f, m, aggregate=True):
    """(fused, separate) results of one Multi-Krum call."""
    gf.set_fused(True)
    a = gf.multikrum(xt, f, m, aggregate=aggregate)
    gf.set_fused(False)
    try:
        b = gf.multikrum(xt, f, m, aggregate=aggregate)
    finally:
        gf.set_fused(True)
    return a, b


def _launched(fn):
    """Kernel names one call launches (per-kernel timing on around it)."""
    gf.set_kernel_timing(True)
    try:
        fn()
        return set(gf.kernel_timing())
    finally:
        gf.set_kernel_timing(False)


def _same(a, b):
    if isinstance(a, tuple):
        return all(_same(u, v) for u, v in zip(a, b))
    if a is None or b is None:
        return a is None and b is None
    return torch.equal(a, b)


@pytest.mark.parametrize("n", [3, 4, 5, 7, 8, 11, 12])
@pytest.mark.parametrize("d", [1, 3, 1000, 1024, 1025, 4099, 100000, 129024, 228352])
def test_fused_equals_separate_kernels(n, d):
    rng = np.random.default_rng(n * 100003 + d)
    x = rng.standard_normal((n, d)).astype(np.float32)
    x[: n // 3] *= 4.0
    xt = _to_dev(x)
    fmax = (n - 3) // 2
    for f in sorted({0, fmax}):
        for m in sorted({1, max(1, (n - f) // 2), n - f}):
            a, b = _both(xt, f, m)
            assert _same(a, b), (n, d, f, m)
            sa, sb = _both(xt, f, m, aggregate=False)  # selection only
            assert sa[0] is None and torch.equal(sa[1], a[1]), (n, d, f, m)
            assert torch.equal(sb[1], a[1]), (n, d, f, m)


def test_short_inputs_take_two_launches():
    w = synth.WORKLOADS[1]
    xt = synth.generate(w, DEV).x
    names = _launched(lambda: gf.krum(xt, w.f))
    assert names == {"dist_direct", "krum_select_mean"}, names
    # more partials than the combined kernel reads again, n > 12, or no
    # output: the separate kernels
    for shape, aggregate in (((7, 300000), True), ((13, 1000), True), ((7, 1000), False)):
        x = torch.zeros(shape, device=DEV)
        names = _launched(lambda: gf.multikrum(x, 1, 1, aggregate=aggregate))
        assert "krum_select_mean" not in names and "krum_select" in names, (shape, names)


def test_workload_shape_against_oracle():
    # the n = 7, f = 1, d = 100,000 workload itself, and Multi-Krum on it
    w = synth.WORKLOADS[1]
    for t in range(10):
        inp = synth.generate(w, "cpu", seed=w.seed + t)
        x = inp.x.numpy()
        xt = _to_dev(x)
        Do = oracle.pairwise_sqdist(x)
        B = parity.dist_bounds(Do, "direct")
        same = parity.identical_rows(Do)
        oo, so, sc = oracle.multikrum(x, w.f, 1, return_scores=True)
        if not parity.krum_pinned(sc, Do, B, w.f, 1, same)[0]:
            continue
        out, sel = gf.krum(xt, w.f)
        assert sel.cpu().tolist() == so.tolist()
        assert np.array_equal(out.cpu().numpy(), oo)
        assert np.array_equal(oo, x[so[0]])
        for m in (2, 4, w.n - w.f):
            oo, so, sc = oracle.multikrum(x, w.f, m, return_scores=True)
            assert parity.krum_pinned(sc, Do, B, w.f, m, same)[0], m
            out, sel = gf.multikrum(xt, w.f, m)
            assert sel.cpu().tolist() == so.tolist(), m
            ok, at, err = parity.agg_close(out.cpu().numpy(), oo)
            assert ok, (m, at, err)
        return
    pytest.fail("no pinned seed in 10 tries")


def test_small_integer_ties_against_oracle():
    # exact distances on both sides: every tie goes to the lower index
    rng = np.random.default_rng(11)
    for trial in range(25):
        n = int(rng.integers(3, 13))
        d = int(rng.choice([33, 2000, 70001]))
        x = rng.integers(-2, 3, size=(n, d)).astype(np.float32)
        xt = _to_dev(x)
        for f in range(0, (n - 3) // 2 + 1):
            for m in sorted({1, n - f}):
                out, sel = gf.multikrum(xt, f, m)
                oo, so = oracle.multikrum(x, f, m)
                assert sel.cpu().tolist() == so.tolist(), (trial, n, d, f, m)
                assert np.array_equal(out.cpu().numpy(), oo), (trial, n, d, f, m)


def test_consecutive_calls_of_other_shapes():
    # the partials of one call never leak into the next (other tile counts)
    rng = np.random.default_rng(12)
    shapes = [(7, 100000), (7, 5000), (12, 129024), (5, 1), (7, 100000), (9, 150001)]
    xs = [_to_dev(rng.standard_normal(s).astype(np.float32)) for s in shapes]
    want = []
    gf.set_fused(False)
    try:
        for xt in xs:
            want.append(gf.multikrum(xt, 1, 2))
    finally:
        gf.set_fused(True)
    for rep in range(3):
        for xt, (wo, ws) in zip(xs, want):
            out, sel = gf.multikrum(xt, 1, 2)
            assert torch.equal(sel, ws) and torch.equal(out, wo), (rep, tuple(xt.shape))


def test_unaligned_input_rows():
    # rows only 4-byte aligned (a view one float into its storage)
    rng = np.random.default_rng(13)
    for d in (10006, 10007):
        base = _to_dev(rng.standard_normal(11 * d + 1).astype(np.float32))
        xt = base[1:].view(11, d)
        a, b = _both(xt, 2, 9)
        assert _same(a, b), d
        a, b = _both(xt, 2, 1)
        assert _same(a, b), d
