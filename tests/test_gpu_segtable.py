"""GPU parity of segment tables: vectors stored apart, aggregated per segment.

Each vector's segments are separate allocations (some one float into their
buffer, so 4-byte but not 16-byte aligned), with ragged lengths including
empty and one-float segments, and more segments than one launch takes (96),
so a batch spans several launches. Checks:

* the selection equals the oracle's on the concatenated vectors whenever
  every decision is pinned (the bound of the summed distances is the sum of
  the segments' direct-engine bounds), and each segment's aggregate is within
  max(1e-5 |oracle|, 1e-6) of the oracle's on that segment's coordinates
  (bit-exact for Krum and Median);
* each segment's aggregate equals, bit for bit, the matrix-based segmented
  session's aggregate of the same segment (the same per-coordinate code; only
  the addressing differs);
* K = 1 (n whole vectors in separate buffers) reproduces the plain rule on
  the stacked matrix bit for bit: the same tiles, summed in the same order;
* n > 20 (the Gram engine over the table): the selection equals the oracle's
  when pinned under the Gram bound for the table's own reference row, and the
  aggregates are within the same tolerance (bit-exact for Krum and Median).
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
    gf.set_direct_max_n(20)


def _split(d, K, rng):
    """K ragged segment lengths summing to d, with an empty and a one-float one."""
    cuts = np.sort(rng.choice(np.arange(1, d), size=K - 1, replace=False))
    sizes = np.diff(np.concatenate([[0], cuts, [d]])).tolist()
    sizes[1], sizes[2] = 0, 1  # keep the total: move the mass to the last segment
    sizes[-1] += d - sum(sizes)
    return sizes


def _stored_apart(x, sizes, rng):
    """vectors[i][s]: segment s of vector i in its own buffer (some misaligned)."""
    n = x.shape[0]
    cuts = np.concatenate([[0], np.cumsum(sizes)])
    vectors, keep = [], []
    for i in range(n):
        row = []
        for s, (a, b) in enumerate(zip(cuts[:-1], cuts[1:])):
            off = int(rng.integers(0, 2))
            buf = torch.empty(int(b - a) + off, dtype=torch.float32, device=DEV)
            seg = buf[off:]
            seg.copy_(torch.from_numpy(np.ascontiguousarray(x[i, a:b])))
            row.append(seg)
            keep.append(buf)
        vectors.append(row)
    return vectors, keep


def _oracle(rule, x, f, m):
    if rule == "krum":
        return oracle.krum(x, f)
    if rule == "multikrum":
        return oracle.multikrum(x, f, m)
    if rule == "multikrum_iterated":
        return oracle.multikrum_iterated(x, f, m)
    if rule == "bulyan":
        return oracle.bulyan(x, f)
    if rule == "mda":
        return oracle.mda(x, f)
    if rule == "median":
        return oracle.median(x, f), None
    return (x.astype(np.float64).sum(0) / x.shape[0]).astype(np.float32), None


def _pinned(rule, x, f, m, D, B):
    same = parity.identical_rows(D)
    if rule in ("krum", "multikrum"):
        _, _, sc = oracle.multikrum(x, f, m, return_scores=True)
        return parity.krum_pinned(sc, D, B, f, m, same)[0]
    if rule in ("bulyan", "multikrum_iterated"):
        fn = oracle.bulyan if rule == "bulyan" else (lambda a, b, **k: oracle.multikrum_iterated(a, b, m, **k))
        _, _, picks, rs = fn(x, f, return_rounds=True)
        return parity.bulyan_pinned(picks, rs, D, B, x.shape[0], f, same)[0]
    if rule == "mda":
        _, so = oracle.mda(x, f)
        return parity.mda_pinned(D, B, x.shape[0], f, so)[0]
    return True


CASES = [("krum", 1), ("median", 1), ("multikrum", 2), ("multikrum_iterated", 6), ("bulyan", 3),
         ("mda", 4), ("average", 2)]


@pytest.mark.parametrize("rule,key", CASES)
def test_table_equals_concatenated_and_matrix_sessions(rule, key):
    w = synth.WORKLOADS[key]
    n, f = w.n, w.f
    m = {"krum": 1, "multikrum": w.m, "multikrum_iterated": w.m}.get(rule)
    d, K = 30011, 130
    for attempt in range(5):
        seed = w.seed + 7 * attempt
        rng = np.random.default_rng(seed)
        x = synth.generate(w, "cpu", d=d, seed=seed).x.numpy()
        sizes = _split(d, K, rng)
        D = oracle.pairwise_sqdist(x)
        cuts = np.concatenate([[0], np.cumsum(sizes)])
        B = np.zeros((n, n))
        for a, b in zip(cuts[:-1], cuts[1:]):
            if b > a:
                B += parity.dist_bounds(oracle.pairwise_sqdist(x[:, a:b]), "direct")
        if not _pinned(rule, x, f, m, D, B):
            continue
        vectors, keep = _stored_apart(x, sizes, rng)
        table = gf.SegmentTable(vectors)
        seg = gf.Segmented(rule, n, f, m)
        mat = gf.Segmented(rule, n, f, m)
        try:
            for step in range(2):  # the second step checks reset
                seg.reset()
                seg.accumulate_table(table)
                sel = seg.select()
                outs = seg.aggregate_table(table)
                want, want_sel = _oracle(rule, x, f, m)
                if want_sel is not None:
                    assert sel.cpu().numpy().tolist() == want_sel.tolist(), (rule, seed, step)
                got = torch.cat(outs).cpu().numpy()
                if rule in ("krum", "median"):
                    assert np.array_equal(got, want), (rule, seed)
                else:
                    ok, at, err = parity.agg_close(got, want)
                    assert ok, (rule, seed, at, err)
            # the matrix-based session on the same segments: same aggregates, bit for bit
            xt = torch.from_numpy(x).to(DEV)
            mats = [xt[:, a:b].contiguous() for a, b in zip(cuts[:-1], cuts[1:])]
            mat.reset()
            for s_ in mats:
                mat.accumulate(s_)
            msel = mat.select()
            if msel is not None:
                assert msel.cpu().tolist() == sel.cpu().tolist()
            for o, s_ in zip(outs, mats):
                assert torch.equal(o, mat.aggregate(s_)), rule
        finally:
            seg.close()
            mat.close()
        return
    pytest.fail(f"{rule}: no pinned seed in 5 tries")


@pytest.mark.parametrize("rule,n,f", [("multikrum", 11, 2), ("bulyan", 19, 4), ("mda", 10, 3),
                                      ("median", 20, 3), ("krum", 7, 1), ("multikrum", 13, 3)])
def test_row_pointer_form_equals_the_plain_rule(rule, n, f):
    rng = np.random.default_rng(n * 10 + f)
    d = 70001
    x = (rng.standard_normal((n, d)) * np.linspace(0.5, 2.0, n)[:, None]).astype(np.float32)
    rows = []
    for i in range(n):
        buf = torch.empty(d + 1, dtype=torch.float32, device=DEV)
        rows.append(buf[i % 2:i % 2 + d])
        rows[-1].copy_(torch.from_numpy(x[i]))
    table = gf.SegmentTable.rows(rows)
    seg = gf.Segmented(rule, n, f)
    try:
        seg.accumulate_table(table)
        sel = seg.select()
        (out,) = seg.aggregate_table(table)
    finally:
        seg.close()
    xt = torch.from_numpy(x).to(DEV)
    want, want_sel = gf.gar(rule, xt, f)
    assert torch.equal(out, want)
    if want_sel is not None:
        assert torch.equal(sel, want_sel)


def test_many_tiny_segments():
    # 300 segments of 1..40 floats: latency-bound on the per-segment path
    n, f = 11, 2
    rng = np.random.default_rng(77)
    sizes = rng.integers(1, 41, size=300).tolist()
    d = int(sum(sizes))
    x = rng.standard_normal((n, d)).astype(np.float32)
    x[:2] *= 30.0
    vectors, keep = _stored_apart(x, sizes, rng)
    table = gf.SegmentTable(vectors)
    seg = gf.Segmented("multikrum", n, f)
    try:
        seg.accumulate_table(table)
        sel = seg.select()
        got = torch.cat(seg.aggregate_table(table)).cpu().numpy()
    finally:
        seg.close()
    want, want_sel = oracle.multikrum(x, f)
    assert sel.cpu().numpy().tolist() == want_sel.tolist()
    ok, at, err = parity.agg_close(got, want)
    assert ok, (at, err)


GRAM_CASES = [("multikrum", 33, 7, 26), ("krum", 64, 15, 1), ("multikrum_iterated", 33, 7, 9),
              ("bulyan", 27, 6, None), ("mda", 23, 2, None), ("median", 40, 9, None),
              ("average", 21, 0, None)]


@pytest.mark.parametrize("rule,n,f,m", GRAM_CASES)
def test_gram_table_matches_the_oracle(rule, n, f, m):
    # n > 20: the Gram engine over the table (one reference row for every
    # segment), ragged and misaligned segments over more than one launch
    d, K = 40009, 110
    for attempt in range(5):
        rng = np.random.default_rng(1000 * n + f + 17 * attempt)
        x = (rng.standard_normal((n, d)) * (1.0 + 0.5 * rng.permutation(n)[:, None] / n)).astype(np.float32)
        x[:f] *= 8.0
        sizes = _split(d, K, rng)
        vectors, keep = _stored_apart(x, sizes, rng)
        table = gf.SegmentTable(vectors)
        D = oracle.pairwise_sqdist(x)
        # the table's reference row is probed on its longest segment (the first
        # of equal ones); checked against the probe rule on that segment
        big = int(np.argmax(sizes))
        off = int(sum(sizes[:big]))
        ref = parity.checked_reference(np.ascontiguousarray(x[:, off:off + sizes[big]]),
                                       gf.table_gram_reference(table))
        B = parity.dist_bounds(D, "gram", ref, x, segments=sizes)
        if not _pinned(rule, x, f, m, D, B):
            continue
        seg = gf.Segmented(rule, n, f, m)
        try:
            seg.accumulate_table(table)
            sel = seg.select()
            got = torch.cat(seg.aggregate_table(table)).cpu().numpy()
        finally:
            seg.close()
        want, want_sel = _oracle(rule, x, f, m)
        if want_sel is not None:
            assert sel.cpu().numpy().tolist() == want_sel.tolist(), (rule, attempt)
        if rule in ("krum", "median"):
            assert np.array_equal(got, want), rule
        else:
            ok, at, err = parity.agg_close(got, want)
            assert ok, (rule, at, err)
        return
    pytest.fail(f"{rule}: no pinned seed in 5 tries")


def test_gram_table_identical_rows_tie_by_index():
    # identical vectors in different 16-row blocks get identical distance rows
    n, f, d = 40, 9, 9001
    rng = np.random.default_rng(3)
    x = rng.standard_normal((n, d)).astype(np.float32)
    x[37] = x[2]
    x[38] = x[2]
    vectors, keep = _stored_apart(x, _split(d, 12, rng), rng)
    seg = gf.Segmented("multikrum", n, f, 1)
    try:
        seg.accumulate_table(gf.SegmentTable(vectors))
        sel = seg.select().cpu().tolist()
    finally:
        seg.close()
    want = oracle.multikrum(x, f, 1)[1].tolist()
    assert sel == want


def test_table_validation():
    y = torch.zeros((7, 8), dtype=torch.float32, device=DEV)
    seg = gf.Segmented("multikrum", 7, 1)
    try:
        t = gf.SegmentTable.rows(list(y))
        with pytest.raises(gf.GarfieldError) as e:
            seg.aggregate_table(t)  # before any selection
        assert e.value.code == gf.EINVAL
        lib = gf.load()
        import ctypes
        bad = (ctypes.c_int64 * 1)(-1)
        assert lib.garfield_seg_accumulate_table(seg._h, ctypes.c_void_p(t.ptrs.data_ptr()), bad, 1,
                                                 None) == gf.EINVAL
        assert lib.garfield_seg_aggregate_table(seg._h, ctypes.c_void_p(t.ptrs.data_ptr()), t._dims,
                                                1, None, None) == gf.EINVAL
    finally:
        seg.close()
