"""Garfield's robust gradient aggregation rules on MI355X (gfx950).

Thin Python binding over ``libgarfield.so`` (C-ABI declared in
``include/garfield.h``). It only marshals arguments: every step of every rule
runs in the library's HIP kernels. PyTorch provides device memory (the input
and output tensors) and the current stream; nothing here computes on the
tensors. The interface mirrors the paper's ``init()`` / ``aggregate()`` pair
(Section 3.2, Aggregation): ``gar(name, x, f)`` aggregates the n rows of an
``n x d`` fp32 CUDA/HIP tensor.

If the library has not been built, every call raises ``LibraryMissing``; there
is no fallback implementation.
"""
from __future__ import annotations

import ctypes
import os

import torch  # first: libgarfield must bind to the HIP runtime torch has loaded

__all__ = [
    "GarfieldError", "LibraryMissing", "library_path", "load",
    "pairwise_sqdist", "krum", "multikrum", "multikrum_iterated", "median", "bulyan", "mda",
    "average",
    "multikrum_median", "gar", "workspace_bytes", "release", "set_direct_max_n",
    "distance_engine", "gram_reference", "table_gram_reference", "stream_read", "set_kernel_timing", "kernel_timing", "RULES",
    "ATTACKS", "attack", "variance_stats", "delta", "variance_condition", "Segmented",
    "SegmentTable", "contract_step", "contract",
]

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libgarfield.so")

OK, EINVAL, EREQ, ETOOBIG, ENOMEM, EHIP = range(6)
RULE_IDS = {"dist": 0, "krum": 1, "multikrum": 2, "median": 3, "bulyan": 4, "mda": 5, "average": 6,
            "multikrum_iterated": 7}
ATTACKS = {"reverse": 0, "random": 1, "little": 2, "empire": 3}
NMAX = 64


class LibraryMissing(RuntimeError):
    pass


class GarfieldError(RuntimeError):
    def __init__(self, code: int, where: str, message: str):
        super().__init__(f"{where}: {message} (status {code})")
        self.code = code


_lib = None


def library_path() -> str:
    return _LIB_PATH


def load():
    """Load libgarfield.so (raises LibraryMissing if it is not built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(_LIB_PATH):
        raise LibraryMissing(
            f"{_LIB_PATH} is not built; run `python -c 'import __graft_entry__ as g; g.build()'`")
    lib = ctypes.CDLL(_LIB_PATH)
    vp, i32, i64 = ctypes.c_void_p, ctypes.c_int, ctypes.c_int64
    st = ctypes.c_int
    sig = {
        "garfield_pairwise_sqdist": [vp, i32, i64, vp, vp],
        "garfield_krum": [vp, i32, i32, i64, vp, vp, vp],
        "garfield_multikrum": [vp, i32, i32, i64, i32, vp, vp, vp],
        "garfield_multikrum_noalloc": [vp, i32, i32, i64, i32, vp, vp, vp],
        "garfield_multikrum_iterated": [vp, i32, i32, i64, i32, vp, vp, vp],
        "garfield_median": [vp, i32, i32, i64, vp, i32, vp, vp],
        "garfield_bulyan": [vp, i32, i32, i64, vp, vp, vp],
        "garfield_mda": [vp, i32, i32, i64, vp, vp, vp],
        "garfield_average": [vp, i32, i64, vp, vp],
    }
    for name, args in sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = st
    pp = ctypes.POINTER(ctypes.c_void_p)
    seg_sig = {
        "garfield_seg_create": [i32, i32, i32, i32, pp],
        "garfield_seg_reset": [vp, vp],
        "garfield_seg_accumulate": [vp, vp, i64, vp],
        "garfield_seg_select": [vp, vp, vp],
        "garfield_seg_aggregate": [vp, vp, i64, vp, vp],
        "garfield_seg_destroy": [vp],
        "garfield_seg_accumulate_table": [vp, vp, vp, i32, vp],
        "garfield_seg_aggregate_table": [vp, vp, vp, i32, vp, vp],
    }
    for name, args in seg_sig.items():
        fn = getattr(lib, name)
        fn.argtypes = args
        fn.restype = st
    lib.garfield_contract_step.argtypes = [i32, vp, i32, i64, vp, i32, i32, i32, vp, vp]
    lib.garfield_contract_step.restype = st
    lib.garfield_attack.argtypes = [i32, vp, i32, i64, ctypes.c_double, ctypes.c_uint64, vp, i32,
                                    vp]
    lib.garfield_attack.restype = st
    lib.garfield_variance_stats.argtypes = [vp, i32, i64, vp, vp, vp]
    lib.garfield_variance_stats.restype = st
    lib.garfield_delta.argtypes = [i32, i32, i32]
    lib.garfield_delta.restype = ctypes.c_double
    lib.garfield_variance_margin.argtypes = [i32, i32, i32, ctypes.POINTER(ctypes.c_double)]
    lib.garfield_variance_margin.restype = ctypes.c_double
    lib.garfield_workspace_bytes.argtypes = [i32, i32, i32, i64, i32]
    lib.garfield_workspace_bytes.restype = ctypes.c_size_t
    lib.garfield_release.argtypes = []
    lib.garfield_release.restype = st
    lib.garfield_strerror.argtypes = [st]
    lib.garfield_strerror.restype = ctypes.c_char_p
    lib.garfield_version.argtypes = []
    lib.garfield_version.restype = ctypes.c_char_p
    lib.garfield_tuning_set_direct_max_n.argtypes = [i32]
    lib.garfield_tuning_set_direct_max_n.restype = i32
    lib.garfield_tuning_set_fused.argtypes = [i32]
    lib.garfield_tuning_set_fused.restype = i32
    lib.garfield_tuning_set_stream_residency.argtypes = [i32]
    lib.garfield_tuning_set_stream_residency.restype = i32
    lib.garfield_tuning_set_mda_cover_min.argtypes = [ctypes.c_longlong]
    lib.garfield_tuning_set_mda_cover_min.restype = ctypes.c_longlong
    lib.garfield_tuning_distance_engine.argtypes = [i32, ctypes.c_longlong]
    lib.garfield_tuning_distance_engine.restype = i32
    lib.garfield_tuning_gram_reference.argtypes = [vp, i32, ctypes.c_longlong, vp]
    lib.garfield_tuning_gram_reference.restype = i32
    lib.garfield_tuning_stream_read.argtypes = [vp, ctypes.c_longlong, vp, vp]
    lib.garfield_tuning_stream_read.restype = i32
    lib.garfield_tuning_table_gram_reference.argtypes = [vp, i32, vp, i32, vp]
    lib.garfield_tuning_table_gram_reference.restype = i32
    lib.garfield_tuning_set_kernel_timing.argtypes = [i32]
    lib.garfield_tuning_set_kernel_timing.restype = i32
    lib.garfield_tuning_kernel_timing.argtypes = [ctypes.c_char_p, ctypes.c_size_t]
    lib.garfield_tuning_kernel_timing.restype = ctypes.c_size_t
    _lib = lib
    return lib


def _check(code: int, where: str):
    if code != OK:
        msg = load().garfield_strerror(code).decode()
        raise GarfieldError(code, where, msg)


def _stream(x: torch.Tensor) -> ctypes.c_void_p:
    return ctypes.c_void_p(torch.cuda.current_stream(x.device).cuda_stream)


def _input(x: torch.Tensor) -> torch.Tensor:
    if not isinstance(x, torch.Tensor) or x.dim() != 2:
        raise ValueError("x must be a 2-D tensor (n vectors of d values)")
    if x.device.type != "cuda":
        raise ValueError("x must be on a GPU: this library has no CPU path")
    if x.dtype != torch.float32:
        raise ValueError("x must be float32")
    if not x.is_contiguous():
        raise ValueError("x must be contiguous (row-major n x d)")
    return x


def _ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else ctypes.c_void_p(0)


def pairwise_sqdist(x: torch.Tensor) -> torch.Tensor:
    """n x n fp64 squared Euclidean distances."""
    x = _input(x)
    n, d = x.shape
    dist = torch.empty((n, n), dtype=torch.float64, device=x.device)
    _check(load().garfield_pairwise_sqdist(_ptr(x), n, d, _ptr(dist), _stream(x)),
           "garfield_pairwise_sqdist")
    return dist


def multikrum(x: torch.Tensor, f: int, m: int | None = None, aggregate: bool = True):
    """(aggregate or None, sel) -- the m <= n-f vectors of lowest Krum score."""
    x = _input(x)
    n, d = x.shape
    mm = (n - f) if (m is None or m <= 0) else m
    sel = torch.empty(max(mm, 1), dtype=torch.int32, device=x.device)
    out = torch.empty(d, dtype=torch.float32, device=x.device) if aggregate else None
    _check(load().garfield_multikrum(_ptr(x), n, f, d, 0 if m is None else m, _ptr(out),
                                     _ptr(sel), _stream(x)), "garfield_multikrum")
    return out, sel[:mm]


def multikrum_iterated(x: torch.Tensor, f: int, m: int | None = None, aggregate: bool = True):
    """(aggregate or None, sel) -- m rounds of Krum, each over the vectors not
    selected yet (Bulyan's selection stopped after m rounds), then their mean."""
    x = _input(x)
    n, d = x.shape
    mm = (n - f) if (m is None or m <= 0) else m
    sel = torch.empty(max(mm, 1), dtype=torch.int32, device=x.device)
    out = torch.empty(d, dtype=torch.float32, device=x.device) if aggregate else None
    _check(load().garfield_multikrum_iterated(_ptr(x), n, f, d, 0 if m is None else m, _ptr(out),
                                              _ptr(sel), _stream(x)),
           "garfield_multikrum_iterated")
    return out, sel[:mm]


def krum(x: torch.Tensor, f: int):
    """(aggregate, sel[1]) -- the vector of lowest Krum score."""
    x = _input(x)
    n, d = x.shape
    sel = torch.empty(1, dtype=torch.int32, device=x.device)
    out = torch.empty(d, dtype=torch.float32, device=x.device)
    _check(load().garfield_krum(_ptr(x), n, f, d, _ptr(out), _ptr(sel), _stream(x)),
           "garfield_krum")
    return out, sel


def median(x: torch.Tensor, f: int = 0, rows: torch.Tensor | None = None) -> torch.Tensor:
    """Coordinate-wise median over all rows, or over `rows` (device int32)."""
    x = _input(x)
    n, d = x.shape
    k = n
    if rows is not None:
        if rows.device != x.device or rows.dtype != torch.int32 or rows.dim() != 1:
            raise ValueError("rows must be a 1-D int32 tensor on x's device")
        rows = rows.contiguous()
        k = rows.numel()
    out = torch.empty(d, dtype=torch.float32, device=x.device)
    _check(load().garfield_median(_ptr(x), n, f, d, _ptr(rows), k, _ptr(out), _stream(x)),
           "garfield_median")
    return out


def bulyan(x: torch.Tensor, f: int):
    """(aggregate, sel[n-2f])."""
    x = _input(x)
    n, d = x.shape
    sel = torch.empty(max(n - 2 * f, 1), dtype=torch.int32, device=x.device)
    out = torch.empty(d, dtype=torch.float32, device=x.device)
    _check(load().garfield_bulyan(_ptr(x), n, f, d, _ptr(out), _ptr(sel), _stream(x)),
           "garfield_bulyan")
    return out, sel[: max(n - 2 * f, 0)]


def mda(x: torch.Tensor, f: int, aggregate: bool = True):
    """(aggregate or None, sel[n-f])."""
    x = _input(x)
    n, d = x.shape
    sel = torch.empty(max(n - f, 1), dtype=torch.int32, device=x.device)
    out = torch.empty(d, dtype=torch.float32, device=x.device) if aggregate else None
    _check(load().garfield_mda(_ptr(x), n, f, d, _ptr(out), _ptr(sel), _stream(x)),
           "garfield_mda")
    return out, sel[: max(n - f, 0)]


def average(x: torch.Tensor) -> torch.Tensor:
    x = _input(x)
    n, d = x.shape
    out = torch.empty(d, dtype=torch.float32, device=x.device)
    _check(load().garfield_average(_ptr(x), n, d, _ptr(out), _stream(x)), "garfield_average")
    return out


def multikrum_median(x: torch.Tensor, f: int, m: int | None = None):
    """Multi-Krum selection, then the coordinate-wise median of the selected
    rows (the selection stays on the device and feeds the median directly)."""
    _, sel = multikrum(x, f, m, aggregate=False)
    return median(x, f, rows=sel), sel


RULES = {
    "krum": lambda x, f, **kw: krum(x, f),
    "multikrum": lambda x, f, m=None, **kw: multikrum(x, f, m),
    "multikrum_iterated": lambda x, f, m=None, **kw: multikrum_iterated(x, f, m),
    "median": lambda x, f, rows=None, **kw: (median(x, f, rows), None),
    "bulyan": lambda x, f, **kw: bulyan(x, f),
    "mda": lambda x, f, **kw: mda(x, f),
    "average": lambda x, f=0, **kw: (average(x), None),
    "multikrum-median": lambda x, f, m=None, **kw: multikrum_median(x, f, m),
}


def gar(name: str, x: torch.Tensor, f: int, **kw):
    """Aggregate the rows of x with rule `name`; returns (aggregate, selected indices or None)."""
    try:
        rule = RULES[name]
    except KeyError:
        raise ValueError(f"unknown rule {name!r}; known: {sorted(RULES)}") from None
    return rule(x, f, **kw)


def contract_step(rule: str, x: torch.Tensor, peers: torch.Tensor, f: int, m: int | None = None,
                  out: torch.Tensor | None = None) -> torch.Tensor:
    """One contraction step: row v of the result is `rule` applied to the rows
    peers[v] of x (n nodes, q peers each; peers a device int32 n x q tensor)."""
    x = _input(x)
    n, d = x.shape
    if (not isinstance(peers, torch.Tensor) or peers.dtype != torch.int32 or peers.dim() != 2
            or peers.shape[0] != n or peers.device != x.device):
        raise ValueError("peers must be an n x q int32 tensor on x's device")
    peers = peers.contiguous()
    if out is None:
        out = torch.empty_like(x)
    elif out.shape != x.shape or out.dtype != torch.float32 or not out.is_contiguous():
        raise ValueError("out must be a contiguous n x d float32 tensor")
    _check(load().garfield_contract_step(RULE_IDS[rule], _ptr(x), n, d, _ptr(peers),
                                         peers.shape[1], f, m or 0, _ptr(out), _stream(x)),
           "garfield_contract_step")
    return out


def contract(rule: str, x: torch.Tensor, peers: torch.Tensor, f: int, steps: int,
             m: int | None = None) -> torch.Tensor:
    """`steps` contraction steps from x (x itself is not modified)."""
    a = _input(x).clone()
    b = torch.empty_like(a)
    for _ in range(steps):
        contract_step(rule, a, peers, f, m, out=b)
        a, b = b, a
    return a


def attack(kind: str, honest: torch.Tensor | None, nbyz: int, param: float, seed: int = 0,
           d: int | None = None, out: torch.Tensor | None = None) -> torch.Tensor:
    """nbyz Byzantine vectors (nbyz x d) from the honest rows (h x d): "reverse"
    (param * honest[b % h]), "random" (param * N(0, 1); honest may be None, then
    d or out gives the dimension), "little" (mean - param * std per coordinate)
    or "empire" (-param * mean). `out` (nbyz x d, contiguous fp32 on the same
    device) may be a view into a rule's input, e.g. its last rows."""
    if kind not in ATTACKS:
        raise ValueError(f"unknown attack {kind!r}; known: {sorted(ATTACKS)}")
    if honest is not None:
        honest = _input(honest)
        h, dd = honest.shape
        dev = honest.device
    else:
        if kind != "random":
            raise ValueError(f"attack {kind!r} needs the honest rows")
        h = 0
        dd = d if d is not None else (out.shape[1] if out is not None else None)
        if dd is None:
            raise ValueError("give d or out for a random attack without honest rows")
        dev = out.device if out is not None else torch.device("cuda", torch.cuda.current_device())
    if out is None:
        out = torch.empty((nbyz, dd), dtype=torch.float32, device=dev)
    elif (out.dtype != torch.float32 or out.device != dev or tuple(out.shape) != (nbyz, dd)
          or not out.is_contiguous()):
        raise ValueError("out must be a contiguous nbyz x d fp32 tensor on the input's device")
    s = _stream(out) if honest is None else _stream(honest)
    _check(load().garfield_attack(ATTACKS[kind], _ptr(honest), h, dd, float(param),
                                  seed & 0xFFFFFFFFFFFFFFFF, _ptr(out), nbyz, s),
           "garfield_attack")
    return out


def variance_stats(g: torch.Tensor, grad: torch.Tensor) -> torch.Tensor:
    """Device fp64 [2]: the unbiased estimate of E||g - Eg||^2 over the rows of
    g (from their pairwise distances) and ||grad||^2."""
    g = _input(g)
    h, d = g.shape
    grad = _input(grad.reshape(1, -1)).reshape(-1)
    if grad.numel() != d or grad.device != g.device:
        raise ValueError("grad must hold d values on g's device")
    stats = torch.empty(2, dtype=torch.float64, device=g.device)
    _check(load().garfield_variance_stats(_ptr(g), h, d, _ptr(grad), _ptr(stats), _stream(g)),
           "garfield_variance_stats")
    return stats


def delta(rule: str, n: int, f: int) -> float:
    """Delta of the variance condition (Section 3.1) for "mda", "krum" or
    "median"; NaN for other rules or n below the rule's requirement."""
    return load().garfield_delta(RULE_IDS[rule], n, f)


def variance_condition(g: torch.Tensor, grad: torch.Tensor, n: int, f: int) -> dict:
    """For each rule with a Delta: whether kappa * Delta * sigma <= ||grad||
    can hold for some kappa > 1, i.e. ||grad|| / (Delta * sigma) > 1, with
    sigma estimated from the honest gradient estimates g."""
    stats = variance_stats(g, grad).cpu()
    host = (ctypes.c_double * 2)(float(stats[0]), float(stats[1]))
    res = {"sigma": float(stats[0]) ** 0.5, "grad_norm": float(stats[1]) ** 0.5}  # for display
    for rule in ("mda", "krum", "median"):
        dl = delta(rule, n, f)
        ratio = load().garfield_variance_margin(RULE_IDS[rule], n, f, host)
        res[rule] = {"delta": dl, "ratio": ratio, "holds": ratio > 1.0 if ratio == ratio else None}
    return res


class SegmentTable:
    """n vectors held as K segments stored apart: vectors[i][s] is segment s of
    vector i (a contiguous fp32 tensor on the GPU; every vector's segment s has
    the same number of values). The device table of the K*n pointers is built
    once here; the tensors must stay alive and in place while the table is
    used. `SegmentTable.rows(list of n tensors)` is the K = 1 form: n whole
    vectors in separate buffers."""

    def __init__(self, vectors):
        n = len(vectors)
        if n < 1:
            raise ValueError("no vectors")
        K = len(vectors[0])
        dev = None
        for row in vectors:
            if len(row) != K:
                raise ValueError("every vector needs the same number of segments")
            for t in row:
                if (not isinstance(t, torch.Tensor) or t.device.type != "cuda"
                        or t.dtype != torch.float32 or not t.is_contiguous()):
                    raise ValueError("segments must be contiguous float32 GPU tensors")
                dev = t.device if dev is None else dev
                if t.device != dev:
                    raise ValueError("all segments must be on one device")
        self.dims = [int(vectors[0][s].numel()) for s in range(K)]
        for row in vectors:
            if [int(t.numel()) for t in row] != self.dims:
                raise ValueError("segment s must have the same length in every vector")
        self.n, self.K, self.device = n, K, dev
        self._keep = [list(row) for row in vectors]
        flat = [vectors[i][s].data_ptr() for s in range(K) for i in range(n)]
        self.ptrs = torch.tensor(flat, dtype=torch.int64).to(dev)
        self._dims = (ctypes.c_int64 * max(K, 1))(*self.dims)

    @classmethod
    def rows(cls, vectors):
        return cls([[v.reshape(-1) if v.is_contiguous() else v] for v in vectors])


class Segmented:
    """Segmented aggregation (per-layer, Section 4.2): accumulate the distances
    of segments of the n vectors (each an n x d_s tensor: the same coordinates
    of every vector), select once from their sum, then aggregate every segment
    with that selection. Equal to the rule on the concatenated vectors.

        seg = Segmented("bulyan", n, f)
        for x_s in segments: seg.accumulate(x_s)
        sel = seg.select()
        outs = [seg.aggregate(x_s) for x_s in segments]
        seg.reset()   # next step
    """

    def __init__(self, rule: str, n: int, f: int, m: int | None = None):
        if rule not in ("krum", "multikrum", "multikrum_iterated", "bulyan", "mda", "median",
                        "average"):
            raise ValueError(f"unknown rule {rule!r}")
        self.rule, self.n, self.f = rule, n, f
        mm = (n - f) if not m or m <= 0 else m
        self.count = {"krum": 1, "multikrum": mm, "multikrum_iterated": mm,
                      "bulyan": n - 2 * f, "mda": n - f}.get(rule, 0)
        handle = ctypes.c_void_p()
        _check(load().garfield_seg_create(RULE_IDS[rule], n, f, m or 0, ctypes.byref(handle)),
               "garfield_seg_create")
        self._h = handle

    def _seg(self, x):
        x = _input(x)
        if x.shape[0] != self.n:
            raise ValueError(f"segment has {x.shape[0]} rows, the session {self.n}")
        return x

    def reset(self):
        s = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
        _check(load().garfield_seg_reset(self._h, s), "garfield_seg_reset")

    def accumulate(self, x: torch.Tensor):
        x = self._seg(x)
        _check(load().garfield_seg_accumulate(self._h, _ptr(x), x.shape[1], _stream(x)),
               "garfield_seg_accumulate")

    def select(self, device=None):
        """The selection (device int32, ascending), or None for Median / Average."""
        if self.count == 0:
            return None
        dev = torch.device(device) if device is not None else torch.device("cuda", torch.cuda.current_device())
        sel = torch.empty(self.count, dtype=torch.int32, device=dev)
        s = ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)
        _check(load().garfield_seg_select(self._h, _ptr(sel), s), "garfield_seg_select")
        return sel

    def aggregate(self, x: torch.Tensor) -> torch.Tensor:
        x = self._seg(x)
        out = torch.empty(x.shape[1], dtype=torch.float32, device=x.device)
        _check(load().garfield_seg_aggregate(self._h, _ptr(x), x.shape[1], _ptr(out), _stream(x)),
               "garfield_seg_aggregate")
        return out

    def accumulate_table(self, table: "SegmentTable"):
        """Add the distances of every segment of the table (one launch per 96
        segments)."""
        if table.n != self.n:
            raise ValueError(f"table has {table.n} vectors, the session {self.n}")
        s = ctypes.c_void_p(torch.cuda.current_stream(table.device).cuda_stream)
        _check(load().garfield_seg_accumulate_table(self._h, _ptr(table.ptrs), table._dims,
                                                    table.K, s),
               "garfield_seg_accumulate_table")

    def aggregate_table(self, table: "SegmentTable", outs=None):
        """Aggregate every segment of the table with the session's selection;
        returns the K outputs (or fills `outs`, K contiguous fp32 tensors)."""
        if table.n != self.n:
            raise ValueError(f"table has {table.n} vectors, the session {self.n}")
        if outs is None:
            outs = [torch.empty(dk, dtype=torch.float32, device=table.device) for dk in table.dims]
        elif len(outs) != table.K or any(
                o.numel() != dk or o.dtype != torch.float32 or not o.is_contiguous()
                or o.device != table.device for o, dk in zip(outs, table.dims)):
            raise ValueError("outs must be K contiguous fp32 tensors of the segments' lengths")
        optrs = (ctypes.c_void_p * max(table.K, 1))(*[o.data_ptr() for o in outs])
        s = ctypes.c_void_p(torch.cuda.current_stream(table.device).cuda_stream)
        _check(load().garfield_seg_aggregate_table(self._h, _ptr(table.ptrs), table._dims,
                                                   table.K, optrs, s),
               "garfield_seg_aggregate_table")
        return outs

    def close(self):
        if self._h:
            _check(load().garfield_seg_destroy(self._h), "garfield_seg_destroy")
            self._h = ctypes.c_void_p()

    def __del__(self):
        try:
            if self._h:
                load().garfield_seg_destroy(self._h)
        except Exception:
            pass


def workspace_bytes(rule: str, n: int, f: int, d: int, m: int = 0) -> int:
    return int(load().garfield_workspace_bytes(RULE_IDS[rule], n, f, d, m))


def release():
    _check(load().garfield_release(), "garfield_release")


def set_direct_max_n(n: int) -> int:
    old = load().garfield_tuning_set_direct_max_n(n)
    if old < 0:
        raise ValueError(f"direct_max_n out of range: {n}")
    return old


def set_fused(on: bool) -> bool:
    """Allow (True, the default) or forbid the one-launch Krum / Multi-Krum of
    short inputs; returns the previous setting."""
    return bool(load().garfield_tuning_set_fused(1 if on else 0))


def set_stream_residency(wgs_per_cu: int) -> int:
    """Workgroups per CU of the gathering aggregation kernels (0: automatic,
    < 0: uncapped); returns the previous setting."""
    return int(load().garfield_tuning_set_stream_residency(wgs_per_cu))


def set_mda_cover_min(subsets: int) -> int:
    """MDA searches by vertex covers from this many subsets C(n, f) on, by
    enumeration below; returns the previous threshold."""
    return int(load().garfield_tuning_set_mda_cover_min(subsets))


def gram_reference(x: torch.Tensor) -> int:
    """Row the Gram engine shifts x by (synchronises the current stream)."""
    x = _input(x)
    n, d = x.shape
    ref = load().garfield_tuning_gram_reference(_ptr(x), n, d, _stream(x))
    if ref < 0:
        raise GarfieldError(EHIP, "garfield_tuning_gram_reference", "probe failed")
    return ref


STREAM_READ_BLOCKS = 512  # GARFIELD_TUNING_READ_BLOCKS


def stream_read(x: torch.Tensor, sums: torch.Tensor | None = None) -> torch.Tensor:
    """The plain streaming read of garfield_tuning_stream_read over the
    contiguous fp32 tensor x (16-byte aligned, numel % 4 == 0): returns the
    STREAM_READ_BLOCKS per-workgroup fp32 sums (a bandwidth yardstick)."""
    if not isinstance(x, torch.Tensor) or x.dtype != torch.float32 or not x.is_cuda \
            or not x.is_contiguous():
        raise ValueError("x must be a contiguous float32 device tensor")
    if sums is None:
        sums = torch.empty(STREAM_READ_BLOCKS, dtype=torch.float32, device=x.device)
    _check(load().garfield_tuning_stream_read(_ptr(x), x.numel(), _ptr(sums), _stream(x)),
           "garfield_tuning_stream_read")
    return sums


def table_gram_reference(table: "SegmentTable") -> int:
    """Row the Gram engine (n > 20) shifts a segment table by (synchronises the
    current stream)."""
    ref = load().garfield_tuning_table_gram_reference(
        ctypes.c_void_p(table.ptrs.data_ptr()), table.n, table._dims, table.K,
        ctypes.c_void_p(torch.cuda.current_stream(table.device).cuda_stream))
    if ref < 0:
        raise GarfieldError(EHIP, "garfield_tuning_table_gram_reference", "probe failed")
    return ref


def set_kernel_timing(on: bool) -> bool:
    """Record HIP events around every kernel launch (waits for the device)."""
    return bool(load().garfield_tuning_set_kernel_timing(1 if on else 0))


def kernel_timing() -> dict:
    """{kernel name: (launches, total ms)} since timing was switched on."""
    lib = load()
    size = lib.garfield_tuning_kernel_timing(None, 0) + 1
    buf = ctypes.create_string_buffer(size)
    lib.garfield_tuning_kernel_timing(buf, size)
    out = {}
    for line in buf.value.decode().splitlines():
        name, count, ms = line.split()
        out[name] = (int(count), float(ms))
    return out


def distance_engine(n: int, d: int) -> str:
    return {0: "none", 1: "direct", 2: "gram"}[load().garfield_tuning_distance_engine(n, d)]
