"""The gathers' residency cap (workgroups per CU, set by reserving LDS) only
changes how many workgroups a CU holds: the median and Bulyan's trimmed mean
must write the same bits under every setting (capped paths and uncapped ones
alike: the 16-byte median up to 52 rows, the 8-byte one above, Bulyan's band
and general paths), and match the oracle."""
import numpy as np
import pytest
import torch

import oracle
import paper_2010_05888_amd as gf

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


@pytest.fixture(scope="module", autouse=True)
def _library():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    gf.load()
    yield
    gf.set_stream_residency(0)


def _under_caps(fn):
    outs = []
    for cap in (0, -1, 1, 2, 3, 4, 8):
        old = gf.set_stream_residency(cap)
        try:
            outs.append(fn())
        finally:
            gf.set_stream_residency(old)
    return outs


@pytest.mark.parametrize("k,d", [(7, 100003), (11, 65537), (49, 20011), (64, 4097)])
def test_median_same_bits_under_every_cap(k, d):
    rng = np.random.default_rng(k + d)
    x = rng.standard_normal((k, d)).astype(np.float32)
    xt = torch.from_numpy(x).to(DEV)
    outs = _under_caps(lambda: gf.median(xt, 0))
    for o in outs[1:]:
        assert torch.equal(o, outs[0])
    assert np.array_equal(outs[0].cpu().numpy(), oracle.median(x))


@pytest.mark.parametrize("n,f,d", [(11, 2, 100003), (19, 4, 65537), (35, 8, 20011), (25, 3, 30011)])
def test_bulyan_same_bits_under_every_cap(n, f, d):
    # (25, 3): theta = 19, beta = 13, Bulyan's general path; the others take the band path (beta = 3)
    rng = np.random.default_rng(n * 100 + f)
    x = rng.standard_normal((n, d)).astype(np.float32)
    x *= (1.0 + 0.5 * rng.permutation(n) / n).astype(np.float32)[:, None]
    xt = torch.from_numpy(x).to(DEV)
    outs = _under_caps(lambda: gf.bulyan(xt, f))
    for o, s in outs[1:]:
        assert torch.equal(o, outs[0][0]) and torch.equal(s, outs[0][1])
