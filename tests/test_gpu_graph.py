"""Rule calls captured in a HIP graph (torch.cuda.graph) and replayed.

After a warm-up call has sized the library's workspace, a call enqueues
kernels only (no allocation, no memset node, no host synchronisation), so it
can be captured. Each graph is replayed several times with other eager work
and synchronisations in between, on inputs rewritten between replays, and
every replay must equal the eager call on the same input bit for bit.
"""
import ctypes

import numpy as np
import pytest
import torch

import paper_2010_05888_amd as gf

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


@pytest.fixture(scope="module", autouse=True)
def _library():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    gf.load()


def _call(rule, x, f, out, sel):
    lib = gf.load()
    n, d = x.shape
    s = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    px, po, ps = (ctypes.c_void_p(t.data_ptr()) for t in (x, out, sel))
    if rule == "multikrum":
        return lib.garfield_multikrum(px, n, f, d, 0, po, ps, s)
    if rule == "bulyan":
        return lib.garfield_bulyan(px, n, f, d, po, ps, s)
    if rule == "mda":
        return lib.garfield_mda(px, n, f, d, po, ps, s)
    if rule == "median":
        return lib.garfield_median(px, n, f, d, None, n, po, s)
    if rule == "multikrum_iterated":
        return lib.garfield_multikrum_iterated(px, n, f, d, 3, po, ps, s)
    raise AssertionError(rule)


@pytest.mark.parametrize("rule,n,f,d", [("multikrum", 11, 2, 100003), ("multikrum", 11, 2, 3_000_001),
                                        ("bulyan", 19, 4, 250001), ("mda", 10, 3, 70001),
                                        ("median", 7, 1, 100000), ("multikrum_iterated", 33, 7, 40001)])
def test_graph_replays_equal_eager_calls(rule, n, f, d):
    rng = np.random.default_rng(n + d)
    x = torch.empty((n, d), dtype=torch.float32, device=DEV)
    out = torch.empty(d, dtype=torch.float32, device=DEV)
    sel = torch.zeros(n, dtype=torch.int32, device=DEV)
    inputs = []
    for _ in range(3):
        a = rng.standard_normal((n, d)).astype(np.float32)
        a[:f] *= 10.0
        inputs.append(torch.from_numpy(a).to(DEV))
    x.copy_(inputs[0])
    assert _call(rule, x, f, out, sel) == gf.OK  # warm-up: sizes the workspace
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        assert _call(rule, x, f, out, sel) == gf.OK
    for rep in range(6):
        src = inputs[rep % 3]
        x.copy_(src)
        g.replay()
        torch.cuda.synchronize()
        got, got_sel = out.clone(), sel.clone()
        # eager work between replays: the same call outside the graph
        out2 = torch.empty_like(out)
        sel2 = torch.zeros_like(sel)
        assert _call(rule, x, f, out2, sel2) == gf.OK
        torch.cuda.synchronize()
        assert torch.equal(got, out2), (rule, rep)
        assert torch.equal(got_sel, sel2), (rule, rep)
