"""The exactness rule behind the column-sum mean (no GPU).

The distance pass keeps a coordinate's fp64 column sum only when the exponent
fields of its fp32 values (subnormals counted as 1, zeros ignored) span at most
23 binades: then every running fp64 sum of at most 64 of those values, in any
order, is exact, so subtracting the unselected rows gives the selected rows'
exact sum. Checked here against exact rational sums on values drawn at the
edge of the rule (spreads of exactly 23, subnormals, mixed signs, zeros).
"""
from fractions import Fraction

import numpy as np


def _flag(vals):
    """The rule as the kernel states it, from the largest and smallest nonzero |bits|."""
    b = vals.view(np.uint32) & np.uint32(0x7FFFFFFF)
    nz = b[b != 0]
    if nz.size == 0:
        return True
    emax = int(nz.max() >> 23)
    emin = max(int(nz.min() >> 23), 1)
    return emax < 255 and emax - emin <= 23


def _draw(rng, n, lo_exp, spread):
    """n fp32 values with exponent fields in [lo_exp, lo_exp + spread], full
    random mantissas and signs, some zeros."""
    e = rng.integers(lo_exp, lo_exp + spread + 1, n).astype(np.uint32)
    mant = rng.integers(0, 1 << 23, n).astype(np.uint32)
    sign = rng.integers(0, 2, n).astype(np.uint32) << 31
    v = (sign | (e << 23) | mant).view(np.float32)
    v[rng.random(n) < 0.1] = 0.0
    return v


def _sequential_fp64(vals):
    s = 0.0
    for v in vals:
        s += float(v)
    return s


def test_sums_are_exact_within_23_binades():
    rng = np.random.default_rng(2010)
    checked = 0
    for trial in range(400):
        n = int(rng.integers(2, 65))
        lo = int(rng.choice([1, 2, 60, 100, 127, 200, 231]))
        vals = _draw(rng, n, lo, 23)
        if trial % 5 == 0:  # subnormals among small normals
            k = int(rng.integers(1, n))
            vals[:k] = (rng.integers(1, 1 << 23, k).astype(np.uint32)).view(np.float32)
            vals[k:] = _draw(rng, n - k, 1, 22)
        assert _flag(vals), trial
        exact_total = sum(Fraction(float(v)) for v in vals)
        assert Fraction(_sequential_fp64(vals)) == exact_total
        # the total minus a random subset, as the mean pass forms it
        drop = rng.random(n) < 0.3
        r = _sequential_fp64(vals)
        for v in vals[drop]:
            r -= float(v)
        assert Fraction(r) == sum(Fraction(float(v)) for v in vals[~drop])
        checked += 1
    assert checked == 400


def test_the_rule_rejects_wider_spreads_and_non_finite_values():
    assert not _flag(np.array([1.0, 2.0 ** 24], dtype=np.float32))
    assert _flag(np.array([1.0, 2.0 ** 23 * 1.5], dtype=np.float32))
    assert not _flag(np.array([1.0, np.inf], dtype=np.float32))
    assert _flag(np.zeros(5, dtype=np.float32))
    assert _flag(np.array([0.0, -0.0, 1e-45], dtype=np.float32))
