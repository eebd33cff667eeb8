"""The C-ABI library loads and exports every declared symbol (no GPU needed).

Only calls that the library rejects during host-side validation are made
here: they return before any HIP call, so nothing touches a device.
"""
import ctypes
import os
import re

import pytest

import paper_2010_05888_amd as gf

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = [os.path.join(ROOT, "include", h) for h in ("garfield.h", "garfield_tuning.h")]


def _declared():
    names = set()
    for h in HEADERS:
        text = open(h).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        names.update(re.findall(r"\b(garfield_\w+)\s*\(", text))
    return sorted(names)


def test_headers_declare_the_boundary():
    names = _declared()
    for required in ["garfield_pairwise_sqdist", "garfield_krum", "garfield_multikrum",
                     "garfield_median", "garfield_bulyan", "garfield_mda"]:
        assert required in names


def test_library_exports_every_declared_symbol():
    assert os.path.exists(gf.library_path()), "libgarfield.so is not built"
    lib = ctypes.CDLL(gf.library_path())
    missing = [n for n in _declared() if not hasattr(lib, n)]
    assert not missing, missing


@pytest.fixture(scope="module")
def lib():
    return gf.load()


FAKE = ctypes.c_void_p(0x1000)  # never dereferenced: every call below fails validation
NULL = ctypes.c_void_p(0)


def test_validation_codes(lib):
    # garfield_krum(x, n, f, d, out, sel, stream)
    assert lib.garfield_krum(FAKE, 0, 0, 10, FAKE, FAKE, NULL) == gf.EINVAL
    assert lib.garfield_krum(FAKE, 6, 2, 10, FAKE, FAKE, NULL) == gf.EREQ   # n < 2f+3
    assert lib.garfield_krum(FAKE, 65, 2, 10, FAKE, FAKE, NULL) == gf.ETOOBIG
    assert lib.garfield_krum(NULL, 7, 1, 10, FAKE, FAKE, NULL) == gf.EINVAL
    assert lib.garfield_krum(FAKE, 7, -1, 10, FAKE, FAKE, NULL) == gf.EINVAL
    assert lib.garfield_krum(FAKE, 7, 1, -1, FAKE, FAKE, NULL) == gf.EINVAL
    assert lib.garfield_krum(FAKE, 7, 1, 10, FAKE, NULL, NULL) == gf.EINVAL
    # multikrum: m > n - f
    assert lib.garfield_multikrum(FAKE, 7, 1, 10, 7, FAKE, FAKE, NULL) == gf.EINVAL
    # iterated multikrum: the same requirements
    assert lib.garfield_multikrum_iterated(FAKE, 7, 1, 10, 7, FAKE, FAKE, NULL) == gf.EINVAL
    assert lib.garfield_multikrum_iterated(FAKE, 6, 2, 10, 0, FAKE, FAKE, NULL) == gf.EREQ
    assert lib.garfield_multikrum_iterated(FAKE, 65, 2, 10, 0, FAKE, FAKE, NULL) == gf.ETOOBIG
    assert lib.garfield_multikrum_iterated(FAKE, 7, 1, 10, 0, FAKE, NULL, NULL) == gf.EINVAL
    # median: n < 2f+1, k out of range with a row list, null out
    assert lib.garfield_median(FAKE, 6, 3, 10, NULL, 0, FAKE, NULL) == gf.EREQ
    assert lib.garfield_median(FAKE, 6, 1, 10, FAKE, 7, FAKE, NULL) == gf.EINVAL
    assert lib.garfield_median(FAKE, 6, 1, 10, FAKE, 0, FAKE, NULL) == gf.EINVAL
    assert lib.garfield_median(FAKE, 6, 1, 10, NULL, 0, NULL, NULL) == gf.EINVAL
    # bulyan: n < 4f+3
    assert lib.garfield_bulyan(FAKE, 10, 2, 10, FAKE, FAKE, NULL) == gf.EREQ
    # mda: n < 2f+1, and C(n, f) above the cap
    assert lib.garfield_mda(FAKE, 6, 3, 10, FAKE, FAKE, NULL) == gf.EREQ
    assert lib.garfield_mda(FAKE, 64, 31, 10, FAKE, FAKE, NULL) == gf.ETOOBIG
    # a float pointer that is not 4-byte aligned
    assert lib.garfield_krum(ctypes.c_void_p(0x1002), 7, 1, 10, FAKE, FAKE, NULL) == gf.EINVAL
    assert lib.garfield_median(ctypes.c_void_p(0x1001), 7, 1, 10, NULL, 0, FAKE, NULL) == gf.EINVAL
    # the no-allocation Multi-Krum: the same checks, and sizes whose distance
    # step needs more than its fixed scratch (20 x 2e8: about 74 MB of tile
    # partials) are refused before any HIP call
    assert lib.garfield_multikrum_noalloc(FAKE, 7, 1, 10, 7, FAKE, FAKE, NULL) == gf.EINVAL
    assert lib.garfield_multikrum_noalloc(FAKE, 6, 2, 10, 0, FAKE, FAKE, NULL) == gf.EREQ
    assert lib.garfield_multikrum_noalloc(FAKE, 65, 2, 10, 0, FAKE, FAKE, NULL) == gf.ETOOBIG
    assert lib.garfield_multikrum_noalloc(FAKE, 7, 1, 10, 0, FAKE, NULL, NULL) == gf.EINVAL
    assert lib.garfield_multikrum_noalloc(FAKE, 20, 2, 200_000_000, 0, FAKE, FAKE, NULL) == \
        gf.ETOOBIG
    # distances / average
    assert lib.garfield_pairwise_sqdist(FAKE, 5, 10, NULL, NULL) == gf.EINVAL
    assert lib.garfield_average(FAKE, 0, 10, FAKE, NULL) == gf.EINVAL
    # d beyond one launch ((2^31 - 1) workgroups of 256 coordinates): refused
    # before anything is enqueued, whatever the rule
    huge = (2 ** 31 - 1) * 256 + 1
    assert lib.garfield_average(FAKE, 3, huge, FAKE, NULL) == gf.ETOOBIG
    assert lib.garfield_median(FAKE, 3, 0, huge, NULL, 0, FAKE, NULL) == gf.ETOOBIG
    assert lib.garfield_krum(FAKE, 7, 1, huge, FAKE, FAKE, NULL) == gf.ETOOBIG
    assert lib.garfield_bulyan(FAKE, 7, 1, huge, FAKE, FAKE, NULL) == gf.ETOOBIG


def test_strerror_and_version(lib):
    for code in range(6):
        assert lib.garfield_strerror(code)
    assert b"unknown" in lib.garfield_strerror(99)
    assert lib.garfield_version().startswith(b"garfield")


def test_attack_and_variance_validation(lib):
    A = gf.ATTACKS
    nan = float("nan")
    assert lib.garfield_attack(4, FAKE, 3, 10, 1.0, 0, FAKE, 2, NULL) == gf.EINVAL
    assert lib.garfield_attack(-1, FAKE, 3, 10, 1.0, 0, FAKE, 2, NULL) == gf.EINVAL
    assert lib.garfield_attack(A["little"], FAKE, 3, 10, 1.0, 0, FAKE, 65, NULL) == gf.ETOOBIG
    assert lib.garfield_attack(A["little"], FAKE, 65, 10, 1.0, 0, FAKE, 2, NULL) == gf.ETOOBIG
    assert lib.garfield_attack(A["little"], FAKE, 0, 10, 1.0, 0, FAKE, 2, NULL) == gf.EINVAL
    assert lib.garfield_attack(A["reverse"], NULL, 3, 10, 1.0, 0, FAKE, 2, NULL) == gf.EINVAL
    assert lib.garfield_attack(A["empire"], FAKE, 3, 10, nan, 0, FAKE, 2, NULL) == gf.EINVAL
    assert lib.garfield_attack(A["random"], NULL, 0, 10, 1.0, 0, NULL, 2, NULL) == gf.EINVAL
    assert lib.garfield_attack(A["random"], NULL, 0, -1, 1.0, 0, FAKE, 2, NULL) == gf.EINVAL
    assert lib.garfield_attack(A["little"], FAKE, 3, 10, 1.0, 0, ctypes.c_void_p(0x1002), 2,
                               NULL) == gf.EINVAL
    # nothing to write: accepted without touching the device
    assert lib.garfield_attack(A["little"], FAKE, 3, 10, 1.0, 0, FAKE, 0, NULL) == gf.OK
    assert lib.garfield_attack(A["random"], NULL, 0, 0, 1.0, 0, NULL, 4, NULL) == gf.OK
    # variance statistics: h >= 2, grad and stats required
    assert lib.garfield_variance_stats(FAKE, 1, 10, FAKE, FAKE, NULL) == gf.EINVAL
    assert lib.garfield_variance_stats(FAKE, 3, 10, NULL, FAKE, NULL) == gf.EINVAL
    assert lib.garfield_variance_stats(FAKE, 3, 10, FAKE, NULL, NULL) == gf.EINVAL
    assert lib.garfield_variance_stats(FAKE, 65, 10, FAKE, FAKE, NULL) == gf.ETOOBIG
    # Delta (host closed forms, Section 3.1): n = 11, f = 2
    R = gf.RULE_IDS
    assert lib.garfield_delta(R["median"], 11, 2) == 3.0
    assert lib.garfield_delta(R["krum"], 11, 2) == pytest.approx(36.4 ** 0.5, rel=1e-15)
    assert lib.garfield_delta(R["mda"], 11, 2) == pytest.approx(4 * 2 ** 0.5 / 9, rel=1e-15)
    assert lib.garfield_delta(R["bulyan"], 11, 2) != lib.garfield_delta(R["bulyan"], 11, 2)  # NaN
    assert lib.garfield_delta(R["krum"], 6, 2) != lib.garfield_delta(R["krum"], 6, 2)


def test_workspace_bytes(lib):
    assert gf.workspace_bytes("median", 64, 15, 10 ** 8) == 0
    assert gf.workspace_bytes("krum", 0, 0, 10) == 0
    small = gf.workspace_bytes("multikrum", 11, 2, 11_173_962)
    big = gf.workspace_bytes("multikrum", 64, 15, 138_357_544)
    # n = 11, m = 9: the distance partials plus 8 bytes of column sum per
    # coordinate; m = 7 (2m <= n + 4) has no column sums
    sums = 8 * 11_173_962
    small_m7 = gf.workspace_bytes("multikrum", 11, 2, 11_173_962, 7)
    assert 0 < small_m7 < 4 << 20 and small == small_m7 + (sums + 255) // 256 * 256
    assert 0 < big < 256 << 20
    assert gf.workspace_bytes("mda", 10, 3, 25_557_032) > 0
    assert gf.workspace_bytes("multikrum_iterated", 11, 2, 11_173_962) == small
    assert gf.workspace_bytes("mda", 64, 31, 10) == 0


def test_engine_selection(lib):
    old = gf.set_direct_max_n(20)
    try:
        assert gf.distance_engine(1, 100) == "none"
        assert gf.distance_engine(7, 0) == "none"
        assert gf.distance_engine(19, 100) == "direct"
        assert gf.distance_engine(21, 100) == "gram"
        assert gf.set_direct_max_n(1) == 20
        assert gf.distance_engine(2, 100) == "gram"
        with pytest.raises(ValueError):
            gf.set_direct_max_n(0)
        with pytest.raises(ValueError):
            gf.set_direct_max_n(21)
    finally:
        gf.set_direct_max_n(old)


def test_binding_refuses_cpu_tensors():
    import torch
    with pytest.raises(ValueError):
        gf.krum(torch.zeros((7, 10)), 1)
    with pytest.raises(ValueError):
        gf.median(torch.zeros((7, 10), dtype=torch.float64))


def test_segmented_validation_codes(lib):
    out = ctypes.c_void_p()
    ref = ctypes.byref(out)
    R = gf.RULE_IDS
    assert lib.garfield_seg_create(R["bulyan"], 10, 2, 0, ref) == gf.EREQ    # n < 4f+3
    assert lib.garfield_seg_create(R["krum"], 6, 2, 0, ref) == gf.EREQ      # n < 2f+3
    assert lib.garfield_seg_create(R["multikrum"], 7, 1, 7, ref) == gf.EINVAL  # m > n-f
    assert lib.garfield_seg_create(R["multikrum_iterated"], 7, 1, 7, ref) == gf.EINVAL
    assert lib.garfield_seg_create(R["multikrum_iterated"], 6, 2, 0, ref) == gf.EREQ
    assert lib.garfield_seg_create(R["mda"], 6, 3, 0, ref) == gf.EREQ
    assert lib.garfield_seg_create(R["mda"], 64, 31, 0, ref) == gf.ETOOBIG
    assert lib.garfield_seg_create(R["median"], 5, 3, 0, ref) == gf.EREQ
    assert lib.garfield_seg_create(R["average"], 65, 0, 0, ref) == gf.ETOOBIG
    assert lib.garfield_seg_create(R["dist"], 5, 0, 0, ref) == gf.EINVAL    # not a rule
    assert lib.garfield_seg_create(42, 5, 0, 0, ref) == gf.EINVAL
    assert lib.garfield_seg_create(R["average"], 5, 0, 0, None) == gf.EINVAL
    assert not out.value  # nothing was created
    assert lib.garfield_seg_accumulate(NULL, FAKE, 10, NULL) == gf.EINVAL
    assert lib.garfield_seg_select(NULL, FAKE, NULL) == gf.EINVAL
    assert lib.garfield_seg_aggregate(NULL, FAKE, 10, FAKE, NULL) == gf.EINVAL
    assert lib.garfield_seg_reset(NULL, NULL) == gf.EINVAL
    assert lib.garfield_seg_destroy(NULL) == gf.OK


def test_variance_margin_on_the_host(lib):
    # ||grad|| / (Delta sigma) from host statistics (no GPU): checked against the
    # oracle's Delta; +inf when Delta sigma is 0, NaN without a Delta
    import math

    import oracle

    lib.garfield_variance_margin.argtypes = [ctypes.c_int, ctypes.c_int, ctypes.c_int,
                                             ctypes.POINTER(ctypes.c_double)]
    lib.garfield_variance_margin.restype = ctypes.c_double
    stats = (ctypes.c_double * 2)(0.25, 9.0)  # sigma = 0.5, ||grad|| = 3
    for rule, rid in (("mda", gf.RULE_IDS["mda"]), ("krum", gf.RULE_IDS["krum"]),
                      ("median", gf.RULE_IDS["median"])):
        for n, f in ((7, 1), (11, 2), (19, 4)):
            want = 3.0 / (oracle.delta(rule, n, f) * 0.5)
            assert lib.garfield_variance_margin(rid, n, f, stats) == pytest.approx(want, rel=1e-12)
    zero = (ctypes.c_double * 2)(0.0, 9.0)
    assert math.isinf(lib.garfield_variance_margin(gf.RULE_IDS["median"], 7, 1, zero))
    assert math.isnan(lib.garfield_variance_margin(gf.RULE_IDS["bulyan"], 7, 1, stats))
    assert math.isnan(lib.garfield_variance_margin(gf.RULE_IDS["krum"], 4, 1, stats))  # n < 2f+3
    assert math.isnan(lib.garfield_variance_margin(gf.RULE_IDS["krum"], 7, 1, None))


def test_tuning_switches_on_the_host(lib):
    # host-side settings only: no device is touched
    assert lib.garfield_tuning_set_mda_cover_min(-1) == 1 << 20  # the default, unchanged
    assert lib.garfield_tuning_set_mda_cover_min(5) == 1 << 20
    assert lib.garfield_tuning_set_mda_cover_min(1 << 20) == 5
    assert lib.garfield_tuning_set_fused(0) == 1
    assert lib.garfield_tuning_set_fused(1) == 0
