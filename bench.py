#!/usr/bin/env python3
"""Benchmark one aggregation step on one MI355X and print one JSON line.

Metric: GAR input GB/s = n * d * 4 B / (time of one whole step), with the n x d
input already resident in HBM, plus that rate as a fraction of the 8 TB/s HBM
peak. A step is one full pass of the rule(s) the workload names (distances,
selection and aggregation, all in libgarfield's HIP kernels), launched on
torch's current stream. The default workload is the largest one that fits
one GPU: Multi-Krum (m = 49) and then the Median over its selection, n = 64,
f = 15, d = 138,357,544 (VGG-16-sized vectors, 35.4 GB resident).

Alongside the metric the line carries:
  * roofline: the kernel that took the most time, its algorithmic bytes per
    launch (the rows the rule itself must read and the output it must write)
    divided by its average duration (HIP events stamped by each launch's own
    dispatch, over a separate pass of the same steps); bytes that the design
    adds on top (e.g. column sums written for a later pass) are reported apart
    as design_bytes_per_launch;
  * rooflines: the same figure for every kernel that has an algorithmic byte
    count, and for the Gram distance kernel also its integer matrix-core rate
    (the int8 digit products it executes per launch) against the int8 MFMA
    peak;
  * cpu_baseline: the CPU oracle timed on this host's cores on a bounded
    sample of the same input, with the host's CPU model, its processor count
    and the OpenMP team the oracle ran with.
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

HBM_PEAK_GBS = 8000.0        # MI355X HBM3E, 8 TB/s
INPUT_RING_BYTES = 4 << 30   # inputs smaller than this are alternated between two copies
INT8_MFMA_PEAK_TOPS = 5000.0  # MI355X dense int8 matrix peak, 5.0 POP/s


def _parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=21)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", type=int, default=5, choices=[1, 2, 3, 4, 5, 6],
                    help="1-5: the paper's workload shapes; 6: supplementary, the iterated "
                         "Multi-Krum variant on workload 2's shape")
    ap.add_argument("--all", action="store_true", help="one line per workload (1..6)")
    ap.add_argument("--cpu-seconds", type=float, default=10.0,
                    help="target CPU time of the oracle baseline (0 disables it)")
    ap.add_argument("--direct-max-n", type=int, default=None,
                    help="override the direct/Gram distance engine threshold")
    ap.add_argument("--graph", action="store_true",
                    help="capture each step's launches in a HIP graph and time its replays")
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="time a plain 1 GiB device-to-device copy instead (HBM calibration "
                         "and the reference for the FETCH_SIZE / WRITE_SIZE counters)")
    ap.add_argument("--d", type=int, default=None,
                    help="supplementary run: the workload's rules, n, f and attack at this "
                         "dimension instead (labelled as such in config.workload)")
    ap.add_argument("--segments", type=int, default=1,
                    help="segmented aggregation: the input cut into this many column "
                         "segments held as separate tensors (like per-layer gradients); a "
                         "step accumulates their distances, selects once and aggregates "
                         "each segment (workloads 2-4 and 6)")
    ap.add_argument("--table", action="store_true",
                    help="with --segments: feed the segments as a segment table (vectors stored "
                         "apart; one launch per 96 segments) instead of one call per segment")
    ap.add_argument("--contract", action="store_true",
                    help="contraction steps instead: 20 nodes of ResNet-18 size, each "
                         "aggregating 17 peers (f = 3), one JSON line per rule")
    ap.add_argument("--byzantine", action="store_true",
                    help="the device attack generators and the variance statistics instead: one "
                         "JSON line per case, at workload 3's and 2's shapes")
    ap.add_argument("--fig3", action="store_true",
                    help="the GAR micro-benchmark sweeps of the paper's Fig. 3 instead: one "
                         "JSON line per (GAR, n, d), aggregation time without and with the "
                         "copy of the result to host memory")
    return ap.parse_args()


def calibrate_copy(args):
    """A plain device copy of a known size: achieved HBM rate, and the bytes the
    memory counters should report for it (1 GiB read + 1 GiB written)."""
    import torch

    nbytes = 1 << 30
    src = torch.empty(nbytes // 4, dtype=torch.float32, device="cuda:0").uniform_()
    dst = torch.empty_like(src)
    for _ in range(args.warmup):
        dst.copy_(src)
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for _ in range(args.steps):
        dst.copy_(src)
    end.record()
    torch.cuda.synchronize()
    ms = start.elapsed_time(end) / args.steps
    return {"calibration": "device copy", "bytes_read": nbytes, "bytes_written": nbytes,
            "ms": round(ms, 6), "GBps_read_plus_write": round(2 * nbytes / (ms * 1e-3) / 1e9, 2),
            "steps": args.steps}


def measured_ceiling(steps=20):
    """What this GPU streams in practice, as a yardstick for the kernels'
    achieved bandwidth (the roofline fraction stays against the 8 TB/s peak):
    the library's plain streaming read (garfield_tuning_stream_read) and torch's
    device copy, each over 1 GiB, timed with events after three warm-up runs."""
    import torch

    import paper_2010_05888_amd as gf

    nbytes = 1 << 30
    src = torch.empty(nbytes // 4, dtype=torch.float32, device="cuda:0").fill_(1.0)
    dst = torch.empty_like(src)
    sums = torch.empty(gf.STREAM_READ_BLOCKS, dtype=torch.float32, device="cuda:0")
    out = {}
    for name, fn, moved in (("read_GBps", lambda: gf.stream_read(src, sums), nbytes),
                            ("copy_GBps", lambda: dst.copy_(src), 2 * nbytes)):
        for _ in range(3):
            fn()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(steps):
            fn()
        b.record()
        torch.cuda.synchronize()
        out[name] = round(moved / (a.elapsed_time(b) / steps * 1e-3) / 1e9, 1)
    if abs(float(sums.double().sum()) - nbytes / 4) > 1e-3 * nbytes / 4:
        raise RuntimeError("streaming read returned a wrong sum")
    out["how"] = ("1 GiB: garfield_tuning_stream_read (16-byte nontemporal loads, 512 "
                  "workgroups grid-stride); torch copy_ (read + write counted)")
    del src, dst
    torch.cuda.empty_cache()
    return out


class Step:
    """One aggregation step of a workload with preallocated outputs."""

    def __init__(self, gf, w, x):
        import torch

        self.gf, self.w, self.x = gf, w, x
        self.lib = gf.load()
        n, d = x.shape
        dev = x.device
        self.out = torch.empty(d, dtype=torch.float32, device=dev)
        self.out2 = torch.empty(d, dtype=torch.float32, device=dev)
        self.sel = torch.empty(max(n, 1), dtype=torch.int32, device=dev)
        self.stream = ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)
        p = lambda t: ctypes.c_void_p(t.data_ptr())  # noqa: E731
        self.px, self.pout, self.pout2, self.psel = p(x), p(self.out), p(self.out2), p(self.sel)

    def __call__(self, stream=None):
        lib, w = self.lib, self.w
        n, d = self.x.shape
        f, s = w.f, (stream if stream is not None else self.stream)
        rules = w.rules
        codes = []
        if rules == ("krum", "median"):
            codes.append(lib.garfield_krum(self.px, n, f, d, self.pout, self.psel, s))
            codes.append(lib.garfield_median(self.px, n, f, d, None, n, self.pout2, s))
        elif rules == ("multikrum",):
            codes.append(lib.garfield_multikrum(self.px, n, f, d, w.m, self.pout, self.psel, s))
        elif rules == ("multikrum_iterated",):
            codes.append(lib.garfield_multikrum_iterated(self.px, n, f, d, w.m, self.pout,
                                                         self.psel, s))
        elif rules == ("bulyan",):
            codes.append(lib.garfield_bulyan(self.px, n, f, d, self.pout, self.psel, s))
        elif rules == ("mda",):
            codes.append(lib.garfield_mda(self.px, n, f, d, self.pout, self.psel, s))
        elif rules == ("multikrum-median",):
            codes.append(lib.garfield_multikrum(self.px, n, f, d, w.m, None, self.psel, s))
            codes.append(lib.garfield_median(self.px, n, f, d, self.psel, w.m, self.pout, s))
        else:
            raise ValueError(rules)
        if any(codes):
            raise RuntimeError(f"libgarfield returned {codes}")


def algorithmic(kernel, w):
    """(bound, algorithmic bytes per launch, design bytes per launch) of a kernel
    of workload w. Algorithmic bytes are what the rule itself must move: every
    row the step reads once, the output written once. Design bytes are what
    this kernel actually moves by design when that differs (None otherwise):
    the column sums that the distance pass writes for the complement mean, and
    the complement mean's own reads."""
    n, f, d = w.n, w.f, w.d
    kernel = kernel[:-4] if kernel.endswith("_seg") else kernel  # segment-table forms
    if kernel in ("dist_direct", "dist_gram"):
        return "hbm", 4.0 * n * d, None
    if kernel == "dist_direct_sum":  # the rows; the design also writes one fp64 sum per coordinate
        return "hbm", 4.0 * n * d, 4.0 * n * d + 8.0 * d
    if kernel == "mean_complement":
        # the rule's mean reads the m selected rows and writes the output; this
        # kernel reads the column sums and the n - m unselected rows instead
        return "hbm", 4.0 * (w.m + 1) * d, 8.0 * d + 4.0 * (n - w.m + 1) * d
    if kernel == "mean_rows":
        k = {"krum": 1, "multikrum": w.m, "multikrum_iterated": w.m,
             "mda": n - f}.get(w.rules[0], n)
        return "hbm", 4.0 * (k + 1) * d, None
    if kernel == "krum_select_mean":
        # the rule's mean reads the m selected rows and writes the output; this
        # kernel reads every row's coordinates before the selection is known
        k = 1 if w.rules[0] == "krum" else w.m
        return "hbm", 4.0 * (k + 1) * d, 4.0 * (n + 1) * d
    if kernel == "median":
        k = w.m if w.rules == ("multikrum-median",) else n
        return "hbm", 4.0 * (k + 1) * d, None
    if kernel == "bulyan_agg":
        return "hbm", 4.0 * (n - 2 * f + 1) * d, None
    return None, None, None


def gram_mfma_ops(w):
    """Integer matrix-core operations of one Gram distance launch: every
    16 x 16 block pair of the upper block triangle (NB(NB+1)/2 of them, NB =
    ceil(n / 16)) times 9 products of int8 digits, a multiply and an add each,
    per coordinate (d rounded up to whole 256-coordinate stages)."""
    nb = -(-w.n // 16)
    stages = -(-w.d // 256)
    return float(nb * (nb + 1) // 2 * 256 * 9 * 2) * stages * 256


def source_digest(path):
    """First 16 hex digits of the SHA-256 of a kernel's source file together
    with every header beside it (the per-coordinate bodies, row sources and
    generated networks the kernels share), comments and whitespace removed: it
    changes when the code does, not when a comment does. (String literals
    holding comment markers are not expected in the kernel sources.)"""
    import glob
    import hashlib
    import re

    folder = os.path.dirname(path)
    files = [path] + sorted(glob.glob(os.path.join(folder, "*.h")) +
                            glob.glob(os.path.join(folder, "*.inc")))
    h = hashlib.sha256()
    for name in files:
        with open(name) as fh:
            text = fh.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        text = re.sub(r"\s+", "", text)
        h.update(os.path.basename(name).encode() + b"\0" + text.encode() + b"\0")
    return h.hexdigest()[:16]


def measured_traffic(kernel, key):
    """HBM bytes per launch from the committed counter profile, or None when
    there is none for this kernel and workload or its source code changed since."""
    root = os.path.dirname(os.path.abspath(__file__))
    try:
        with open(os.path.join(root, "profiles", "traffic.json")) as fh:
            entry = json.load(fh).get(f"{kernel}@workload{key}")
        if not entry:
            return None
        digest = source_digest(os.path.join(root, entry["source"]))
        return entry["bytes_per_launch"] if digest == entry["source_sha256"] else None
    except (OSError, KeyError, ValueError):
        return None


def cpu_model():
    """The host CPU's model name, from /proc/cpuinfo."""
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def cpu_baseline(w, x_dev, seconds):
    """Time the oracle on this host on a bounded sample of the input (only the
    sampled coordinates are copied to the host)."""
    import numpy as np

    import oracle

    n, d = x_dev.shape

    def host_slice(width):
        return np.ascontiguousarray(x_dev[:, :width].cpu().numpy())

    # the oracle is O(n^2 d) for distance rules: estimate from a small slice,
    # then run on a slice sized for about `seconds` of CPU work
    def run(xs):
        t = time.perf_counter()
        if w.rules == ("krum", "median"):
            oracle.krum(xs, w.f)
            oracle.median(xs, w.f)
        elif w.rules == ("multikrum",):
            oracle.multikrum(xs, w.f, w.m)
        elif w.rules == ("multikrum_iterated",):
            oracle.multikrum_iterated(xs, w.f, w.m)
        elif w.rules == ("bulyan",):
            oracle.bulyan(xs, w.f)
        elif w.rules == ("mda",):
            oracle.mda(xs, w.f)
        else:
            _, sel = oracle.multikrum(xs, w.f, w.m)
            oracle.median(xs, w.f, rows=sel)
        return time.perf_counter() - t

    probe_d = min(d, 1 << 16)
    t_probe = run(host_slice(probe_d))
    per_coord = max(t_probe / probe_d, 1e-12)
    d_s = int(min(d, max(probe_d, seconds / per_coord)))
    xs = host_slice(d_s)
    reps, total = 0, 0.0
    while reps == 0 or (total < seconds and reps < 50):
        total += run(xs)
        reps += 1
    t = total / reps
    team = oracle.omp_team_size()
    sample = (f"first {d_s} of {d} coordinates" if d_s < d else "the full input") + \
             f", {reps} run(s), mean time {t:.3f} s"
    return {"value": round(n * d_s * 4 / t / 1e9, 4), "unit": "GB/s", "cores": team,
            "kind": "oracle", "sample": sample, "omp_team": team,
            "nproc": len(os.sched_getaffinity(0)), "cpu_count": os.cpu_count(),
            "cpu_model": cpu_model(),
            "scheme": "C++/OpenMP fp64 oracle: the distance pairs split over the team, "
                      "per-coordinate rules over contiguous coordinate shares"}


def bench_workload(key, args):
    import dataclasses

    import torch

    import paper_2010_05888_amd as gf
    from paper_2010_05888_amd import synth

    w = synth.WORKLOADS[key]
    if args.d is not None and args.d != w.d:
        w = dataclasses.replace(w, d=int(args.d),
                                name=f"{w.name} [supplementary: d={int(args.d)}]")
    dev = torch.device("cuda:0")
    print(f"[bench] workload {key}: {w.name}: generating", file=sys.stderr, flush=True)
    inp = synth.generate(w, dev, d=w.d)
    x = inp.x
    # Consecutive steps alternate between two copies of the input when it is
    # small enough for a step to find the previous step's data still in the
    # 256 MB Infinity Cache: every step then starts from HBM, as a step on
    # fresh gradients would. (Reuse within a step is kept.)
    copies = [x] if x.numel() * 4 >= INPUT_RING_BYTES else [x, x.clone()]
    torch.cuda.synchronize()
    if args.segments > 1:
        steps = [SegmentedStep(gf, w, xi, args.segments, args.table) for xi in copies]
        del copies  # the segments are copies of their own
        copies = [None] * len(steps)
        torch.cuda.synchronize()
    else:
        steps = [Step(gf, w, xi) for xi in copies]

    def step_k(k):
        steps[k % len(steps)]()

    for k in range(args.warmup):
        step_k(k)
    torch.cuda.synchronize()
    eager_step_k = step_k
    if args.graph and args.segments > 1:
        raise SystemExit("--graph: plain (unsegmented) workloads only")
    if args.graph:
        # every step's launches captured once into a HIP graph (after the
        # warm-up has sized the library's workspace), then replayed
        graphs = []
        for st in steps:
            g = torch.cuda.CUDAGraph()
            with torch.cuda.graph(g):
                st(stream=ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
            graphs.append(g)
        torch.cuda.synchronize()

        def step_k(k):
            graphs[k % len(graphs)].replay()

        for k in range(args.warmup):
            step_k(k)
        torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    start.record()
    for k in range(args.steps):
        step_k(args.warmup + k)
    end.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = start.elapsed_time(end) / args.steps
    value = w.n * w.d * 4 / (ms * 1e-3) / 1e9
    print(f"[bench] timed {args.steps} steps: {ms:.4f} ms/step (wall {wall * 1e3 / args.steps:.4f})",
          file=sys.stderr, flush=True)

    # second pass: the same steps, each between its own pair of events, for the
    # median and minimum step time (kept out of the timed region above)
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
           for _ in range(args.steps)]
    for k, (a, b) in enumerate(evs):
        a.record()
        step_k(args.warmup + args.steps + k)
        b.record()
    torch.cuda.synchronize()
    per_step = sorted(a.elapsed_time(b) for a, b in evs)
    ms_median = per_step[len(per_step) // 2]
    ms_min = per_step[0]

    # third pass of the same steps with per-kernel HIP events (launched
    # directly: the events are stamped by each kernel's own dispatch)
    gf.set_kernel_timing(True)
    for k in range(args.steps):
        eager_step_k(args.warmup + args.steps + k)
    torch.cuda.synchronize()
    kt = gf.kernel_timing()
    gf.set_kernel_timing(False)
    kernels = {k: {"launches": c, "avg_ms": round(t / c, 6)} for k, (c, t) in kt.items()}
    # the streaming kernel that took the most time (selection kernels have no
    # algorithmic byte count; in latency-bound workloads they can take as long)
    priced = [k for k in kt if algorithmic(k, w)[1]]
    dominant = max(priced or kt, key=lambda k: kt[k][1])
    ceiling = measured_ceiling()

    def kernel_roofline(kern):
        bound, per_launch, design = algorithmic(kern, w)
        if per_launch and args.segments > 1:
            # per-segment calls: one launch per (equal) segment; a segment table: one
            # launch per 96 segments
            per_seg = -(-args.segments // 96) if args.table else args.segments
            per_launch /= per_seg
            design = design / per_seg if design else None
        avg_ms = kt[kern][1] / kt[kern][0]
        r = {"kernel": kern, "bound": bound, "achieved": None, "peak": HBM_PEAK_GBS,
             "unit": "GB/s", "frac": None, "traffic": measured_traffic(kern, key),
             "avg_ms": round(avg_ms, 6), "bytes_per_launch": per_launch}
        if per_launch:
            achieved = per_launch / (avg_ms * 1e-3) / 1e9
            r["achieved"] = round(achieved, 2)
            r["frac"] = round(achieved / HBM_PEAK_GBS, 4)
            r["frac_of_measured_read"] = round(achieved / ceiling["read_GBps"], 4)
        if design:
            r["design_bytes_per_launch"] = design
            r["design_GBps"] = round(design / (avg_ms * 1e-3) / 1e9, 2)
        if kern.startswith("dist_gram") and args.segments == 1:
            ops = gram_mfma_ops(w)
            tops = ops / (avg_ms * 1e-3) / 1e12
            r["mfma"] = {"int8_ops_per_launch": ops, "achieved": round(tops, 1),
                         "peak": INT8_MFMA_PEAK_TOPS, "unit": "TOP/s",
                         "frac": round(tops / INT8_MFMA_PEAK_TOPS, 4)}
        return r

    roofline = kernel_roofline(dominant)
    rooflines = [kernel_roofline(k) for k in sorted(priced, key=lambda k: -kt[k][1])]

    base = None
    if args.cpu_seconds > 0:
        print("[bench] CPU oracle baseline", file=sys.stderr, flush=True)
        base = cpu_baseline(w, x, args.cpu_seconds)

    line = {
        "metric": "GAR input GB/s (n*d*4B/time) and % of HBM peak",
        "value": round(value, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 6),
        "ms_per_step_median": round(ms_median, 6),
        "ms_per_step_min": round(ms_min, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32",
        "data": "synthetic",
        "pct_hbm_peak": round(100 * value / HBM_PEAK_GBS, 2),
        "config": {"workload": w.name + (f" [segmented: {args.segments} segments"
                                          f"{', segment table' if args.table else ''}]"
                                          if args.segments > 1 else ""),
                   "rules": list(w.rules), "n": w.n, "f": w.f, "d": w.d,
                   "m": w.m, "seed": w.seed, "byzantine_rows": inp.byzantine,
                   "distance_engine": gf.distance_engine(w.n, w.d),
                   "launch": "hip graph replay" if args.graph else "direct",
                   "input_copies": len(copies)},
        "kernels": kernels,
        "roofline": roofline,
        "rooflines": rooflines,
        "measured_ceiling": ceiling,
        "cpu_baseline": base,
    }
    del x, inp, steps, copies
    torch.cuda.empty_cache()
    return line


FIG3_N = [7, 11, 15, 19, 23, 27, 31, 35, 39, 47, 55, 63]
FIG3_D = [10**4, 10**5, 10**6, 10**7, 10**8]
FIG3_MDA_MAX_SUBSETS = 250_000_000  # n = 39 (C(39, 9) = 2.1e8) still runs; n = 47 (1.7e10) does not


class SegmentedStep:
    """One step of a workload's rule as a segmented aggregation over `k` column
    segments (separate tensors), with preallocated outputs."""

    RULE = {("multikrum",): "multikrum", ("multikrum_iterated",): "multikrum_iterated",
            ("bulyan",): "bulyan", ("mda",): "mda"}

    def __init__(self, gf, w, x, k, table=False):
        import torch

        if w.rules not in self.RULE:
            raise SystemExit(f"--segments: workload {w.key} has no segmented form")
        self.rule = self.RULE[w.rules]
        n, d = x.shape
        cuts = [d * i // k for i in range(k + 1)]
        self.segs = [x[:, a:b].contiguous() for a, b in zip(cuts[:-1], cuts[1:])]
        self.outs = [torch.empty(s.shape[1], dtype=torch.float32, device=x.device)
                     for s in self.segs]
        self.session = gf.Segmented(self.rule, n, w.f, w.m)
        self.lib = gf.load()
        self.s = ctypes.c_void_p(torch.cuda.current_stream(x.device).cuda_stream)
        p = lambda t: ctypes.c_void_p(t.data_ptr())  # noqa: E731
        self.args = [(p(s), s.shape[1], p(o)) for s, o in zip(self.segs, self.outs)]
        self.table = gf.SegmentTable([[s[i] for s in self.segs] for i in range(n)]) if table else None

    def __call__(self):
        if self.table is not None:
            t, sess = self.table, self.session
            sess.reset()
            sess.accumulate_table(t)
            sess.select()
            sess.aggregate_table(t, outs=self.outs)
            return
        lib, h, s = self.lib, self.session._h, self.s
        codes = [lib.garfield_seg_reset(h, s)]
        for px, d, _ in self.args:
            codes.append(lib.garfield_seg_accumulate(h, px, d, s))
        codes.append(lib.garfield_seg_select(h, None, s))
        for px, d, po in self.args:
            codes.append(lib.garfield_seg_aggregate(h, px, d, po, s))
        if any(codes):
            raise RuntimeError(f"libgarfield returned {codes}")


def fig3_sweep(args):
    """The paper's GAR micro-benchmark (Section 6.3, Fig. 3): aggregation time of
    Average, Median, Multi-Krum (m = n - f), Bulyan and MDA with f = floor((n-3)/4),
    over n at d = 10^7 and over d at n = 17. Inputs: seeded N(0, 1) rows already in
    HBM. Each point is the mean of `steps` calls after `warmup`; "ms_device" times
    the calls alone (events around the batch), "ms_with_copy" each call followed by
    the copy of the aggregate into pinned host memory (as the paper times it)."""
    import math

    import torch

    import paper_2010_05888_amd as gf

    lib = gf.load()
    dev = torch.device("cuda:0")
    s = ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)
    points = [("n", n, 10**7) for n in FIG3_N] + [("d", 17, d) for d in FIG3_D]
    for sweep, n, d in points:
        f = (n - 3) // 4
        g = torch.Generator(device=dev).manual_seed(2010058880 + 1000 * n + int(math.log10(d)))
        x = torch.randn(n, d, device=dev, generator=g)
        out = torch.empty(d, dtype=torch.float32, device=dev)
        host = torch.empty(d, dtype=torch.float32, pin_memory=True)
        sel = torch.empty(n, dtype=torch.int32, device=dev)
        px, po, ps = (ctypes.c_void_p(t.data_ptr()) for t in (x, out, sel))
        calls = {
            "average": lambda: lib.garfield_average(px, n, d, po, s),
            "median": lambda: lib.garfield_median(px, n, f, d, None, n, po, s),
            "multikrum": lambda: lib.garfield_multikrum(px, n, f, d, n - f, po, ps, s),
            "bulyan": lambda: lib.garfield_bulyan(px, n, f, d, po, ps, s),
            "mda": lambda: lib.garfield_mda(px, n, f, d, po, ps, s),
        }
        for name, call in calls.items():
            rec = {"sweep": f"fig3-{sweep}", "gar": name, "n": n, "f": f, "d": d}
            if name == "mda" and math.comb(n, f) > FIG3_MDA_MAX_SUBSETS:
                rec["skipped"] = f"C(n, f) = {math.comb(n, f)} subsets"
                print(json.dumps(rec), flush=True)
                continue
            for _ in range(args.warmup):
                if call():
                    raise RuntimeError(f"libgarfield error in {name}")
            torch.cuda.synchronize()
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            for _ in range(args.steps):
                call()
            b.record()
            torch.cuda.synchronize()
            ms_dev = a.elapsed_time(b) / args.steps
            t0 = time.perf_counter()
            for _ in range(args.steps):
                call()
                host.copy_(out, non_blocking=True)
                torch.cuda.synchronize()
            ms_copy = (time.perf_counter() - t0) * 1e3 / args.steps
            rec.update({"ms_device": round(ms_dev, 5), "ms_with_copy": round(ms_copy, 5),
                        "input_GBps": round(n * d * 4 / (ms_dev * 1e-3) / 1e9, 2)})
            print(json.dumps(rec), flush=True)
        del x, out, host, sel
        torch.cuda.empty_cache()


def byzantine_bench(args):
    """Byzantine vectors (Section 3.2, Main objects; Section 6.5) and the variance
    condition's statistics (Section 3.1, Tradeoffs) at the workloads' shapes:
    the attacks of workload 3 (15 honest rows, 4 Byzantine, ResNet-50 size) and
    workload 2 (2 random rows, ResNet-18 size), and the variance statistics of
    workload 2's 9 honest rows against a true gradient. Each line: mean time of
    `steps` calls after `warmup`, algorithmic bytes (rows read once, rows
    written once) over that time, and the per-kernel HIP-event times."""
    import torch

    import paper_2010_05888_amd as gf

    dev = torch.device("cuda:0")
    cases = [
        ("little", 15, 4, 25_557_032, 1.5), ("empire", 15, 4, 25_557_032, 0.1),
        ("reverse", 15, 4, 25_557_032, -100.0), ("random", 0, 2, 11_173_962, 1.0),
        ("variance", 9, 0, 11_173_962, None),
    ]
    for kind, h, nbyz, d, param in cases:
        g = torch.Generator(device=dev).manual_seed(2010058880 + h + nbyz)
        honest = torch.randn((max(h, 1), d), device=dev, generator=g) * 0.01 if h else None
        if kind == "variance":
            grad = torch.randn(d, device=dev, generator=g) * 0.01
            stats = torch.empty(2, dtype=torch.float64, device=dev)
            lib, s = gf.load(), ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)
            args_ = (ctypes.c_void_p(honest.data_ptr()), h, d, ctypes.c_void_p(grad.data_ptr()),
                     ctypes.c_void_p(stats.data_ptr()), s)

            def call():
                return lib.garfield_variance_stats(*args_)
            nbytes = (h + 1) * d * 4
            label = f"variance statistics h={h} d={d} (workload 2's honest rows + true gradient)"
        else:
            out = torch.empty((nbyz, d), dtype=torch.float32, device=dev)
            lib, s = gf.load(), ctypes.c_void_p(torch.cuda.current_stream(dev).cuda_stream)
            hp = ctypes.c_void_p(honest.data_ptr()) if honest is not None else None
            args_ = (gf.ATTACKS[kind], hp, h, d, float(param), 12345, ctypes.c_void_p(out.data_ptr()),
                     nbyz, s)

            def call():
                return lib.garfield_attack(*args_)
            nbytes = {"little": h + nbyz, "empire": h + nbyz, "reverse": 2 * nbyz,
                      "random": nbyz}[kind] * d * 4
            label = f"attack {kind} param={param} h={h} nbyz={nbyz} d={d}"
        for _ in range(args.warmup):
            if call():
                raise RuntimeError(f"libgarfield error in {label}")
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(args.steps):
            call()
        b.record()
        torch.cuda.synchronize()
        ms = a.elapsed_time(b) / args.steps
        gf.set_kernel_timing(True)
        for _ in range(args.steps):
            call()
        torch.cuda.synchronize()
        kt = gf.kernel_timing()
        gf.set_kernel_timing(False)
        kernels = {k: {"launches": c, "avg_ms": round(t / c, 6)} for k, (c, t) in kt.items()}
        dominant = max(kt, key=lambda k: kt[k][1])
        dom_ms = kt[dominant][1] / kt[dominant][0]
        dom_bytes = nbytes if kind != "variance" else h * d * 4  # the distance pass reads g
        print(json.dumps({
            "bench": "byzantine", "case": label, "ms": round(ms, 5),
            "algorithmic_bytes": nbytes, "GBps": round(nbytes / (ms * 1e-3) / 1e9, 1),
            "pct_hbm_peak": round(100 * nbytes / (ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 1),
            "roofline": {"kernel": dominant, "bound": "hbm", "bytes_per_launch": dom_bytes,
                         "avg_ms": round(dom_ms, 6),
                         "achieved": round(dom_bytes / (dom_ms * 1e-3) / 1e9, 1),
                         "frac": round(dom_bytes / (dom_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)},
            "kernels": kernels, "steps": args.steps, "warmup": args.warmup}), flush=True)
        del honest
        torch.cuda.empty_cache()


def contract_bench(args):
    """Contraction steps (Section 5, decentralized learning): n = 20 nodes of
    ResNet-18 size, each node aggregating q = 17 random peers with f = 3, the
    whole step (distances of all rows once, one selection workgroup per node,
    one aggregation launch for all nodes). Algorithmic bytes: the distance
    pass reads the n rows once; the aggregation reads the n rows once and
    writes the n outputs (8 n d: the nodes share their peers' rows, which the
    launch reads once into L2); `node_bytes` is what the nodes read one by one
    (k rows each, k = q for Median, the selection size otherwise)."""
    import torch

    import paper_2010_05888_amd as gf

    dev = torch.device("cuda:0")
    n, q, f, d = 20, 17, 3, 11_173_962
    g = torch.Generator(device=dev).manual_seed(2010058887)
    x = torch.randn((n, d), device=dev, generator=g) * 0.01
    perm = torch.Generator().manual_seed(2010058887)
    peers = torch.stack([torch.randperm(n, generator=perm)[:q] for _ in range(n)]).to(
        device=dev, dtype=torch.int32)
    y = torch.empty_like(x)
    for rule, m, k in (("median", None, q), ("multikrum", q - f, q - f),
                       ("bulyan", None, q - 2 * f), ("mda", None, q - f)):
        def call():
            gf.contract_step(rule, x, peers, f, m, out=y)
        for _ in range(args.warmup):
            call()
        torch.cuda.synchronize()
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(args.steps):
            call()
        b.record()
        torch.cuda.synchronize()
        ms = a.elapsed_time(b) / args.steps
        gf.set_kernel_timing(True)
        for _ in range(args.steps):
            call()
        torch.cuda.synchronize()
        kt = gf.kernel_timing()
        gf.set_kernel_timing(False)
        agg = {"median": "median_nodes", "multikrum": "mean_nodes", "bulyan": "bulyan_nodes",
               "mda": "mean_nodes"}[rule]
        agg_bytes = 8.0 * n * d
        rows = {agg: agg_bytes}
        if rule != "median":
            rows["dist_direct"] = 4.0 * n * d
        roof = {}
        for kern, nbytes in rows.items():
            if kern in kt:
                kms = kt[kern][1] / kt[kern][0]
                roof[kern] = {"bytes_per_launch": nbytes, "avg_ms": round(kms, 6),
                              "achieved": round(nbytes / (kms * 1e-3) / 1e9, 1),
                              "frac": round(nbytes / (kms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
        print(json.dumps({
            "bench": "contract", "rule": rule, "nodes": n, "peers": q, "f": f, "d": d,
            "ms_per_step": round(ms, 5), "node_bytes": 4.0 * n * (k + 1) * d,
            "GBps_input": round(n * d * 4 / (ms * 1e-3) / 1e9, 1),
            "roofline": roof,
            "kernels": {kk: {"launches": c, "avg_ms": round(t / c, 6)} for kk, (c, t) in kt.items()},
            "steps": args.steps, "warmup": args.warmup}), flush=True)


def main():
    args = _parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py runs on exactly one GPU: the aggregation rules here are a single-GPU "
              "build (no sharding or collectives); run it with --gpus 1", file=sys.stderr)
        sys.exit(2)
    import torch

    import paper_2010_05888_amd as gf

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    if args.calibrate_copy:
        print(json.dumps(calibrate_copy(args)), flush=True)
        return
    gf.load()  # fails loudly when the library is not built
    if args.direct_max_n is not None:
        gf.set_direct_max_n(args.direct_max_n)
    if args.fig3:
        fig3_sweep(args)
        return
    if args.byzantine:
        byzantine_bench(args)
        return
    if args.contract:
        contract_bench(args)
        return
    keys = [1, 2, 3, 4, 5, 6] if args.all else [args.workload]
    for key in keys:
        print(json.dumps(bench_workload(key, args)), flush=True)


if __name__ == "__main__":
    main()
