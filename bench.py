#!/usr/bin/env python3
"""Benchmark of the GETT contraction library on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-report]
                    [--no-cpu-baseline]
    python bench.py --sweep fig11|appendix_a [--max-candidates N] [--report-runs R]

A step is one contraction C <- alpha*A*B + beta*C of the headline workload
(bw4x3_fp32: C[a,b,c,d] = A[a,e,b] * B[e,d,c], a..d = 112, e = 16,
alpha 1.5, beta 1) with inputs already resident in device memory.  W untimed
steps, then K timed steps between device synchronisations; one JSON line on
stdout.  The line also carries:
  roofline      the kernel's algorithmic bytes (or flops) per launch over its
                average launch time (HIP events on the launch stream), against
                MI355X's published peak;
  cpu_baseline  the oracle (plain C, fp64, all host threads) on a bounded
                sample of the same workload;
  workloads     every workload with cold-cache kernel times (minimum and
                median over runs, each after reading a 1 GiB buffer, which
                evicts the workload's data from the caches and leaves no
                dirty lines behind), GFLOP/s,
                GB/s, fraction of its bound, the same contraction by TTGT
                (Sec. 4) and by LoG (Sec. 5), and an equal-size GEMM (torch -> hipBLASLt/rocBLAS)
                timed the same way (Sec. 7: the GEMM of sizes
                S_Im x S_In x S_Ik).
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

import workloads as wl  # noqa: E402

PEAK = {"hbm_GBs": 8000.0, "f32_TFLOPs": 157.3, "f64_TFLOPs": 78.6}
HEADLINE = "bw4x3_fp32"


def log(*a):
    print(*a, file=sys.stderr, flush=True)


# Sources that decide what the GETT kernel does for a given contraction (the
# analyser's plan, the launch and the kernel templates).  The committed HBM
# traffic figure is used only while these are unchanged.
KERNEL_SOURCES = ("analyse.cpp", "api.cpp", "desc.hpp", "direct.hpp", "kernel.hpp", "launch.hpp",
                  "launch_f32.hip", "launch_f64.hip", "plan.hpp", "tiles.hpp")


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_1607_00145_amd", "csrc")
    for f in KERNEL_SOURCES:
        with open(os.path.join(csrc, f), "rb") as fh:
            h.update(f.encode() + fh.read())
    return h.hexdigest()[:16]


def bound_of(w) -> str:
    ai = wl.flop_count(w) / wl.algorithmic_bytes(w)
    ridge = (PEAK["f32_TFLOPs"] if w.dtype == "f32" else PEAK["f64_TFLOPs"]) * 1e3 / PEAK["hbm_GBs"]
    return "mfma" if ai > ridge else "hbm"


class Problem:
    """One workload on the device, planned."""

    def __init__(self, w, dev, on_device: bool = False, flags: int = 0):
        import torch

        import paper_1607_00145_amd as g
        self.w, self.g, self.dev = w, g, dev
        if on_device:
            # timing only: U[-1,1] drawn on the device (seeded), no host copy
            gen = torch.Generator(device=dev)
            gen.manual_seed(w.seed)
            dt = torch.float32 if w.dtype == "f32" else torch.float64
            draw = lambda n: torch.rand(n, generator=gen, dtype=dt, device=dev) * 2 - 1
            self.host = None
            self.A, self.B = draw(w.numel("A")), draw(w.numel("B"))
            self.C0 = draw(w.numel("C")) if w.beta != 0 else None
        else:
            A, B, Cin = wl.make_inputs(w)
            self.host = (A, B, Cin)
            flat = lambda t: torch.from_numpy(np.asfortranarray(t).reshape(-1, order="F")).to(dev)
            self.A, self.B = flat(A), flat(B)
            self.C0 = flat(Cin) if Cin is not None else None
        self.C = self.C0.clone() if self.C0 is not None else torch.zeros(
            w.numel("C"), dtype=self.A.dtype, device=dev)
        dt = g.GETT_FLOAT32 if w.dtype == "f32" else g.GETT_FLOAT64
        st, self.h = g.gett_plan(dt, w.modes_C, w.shape("C"), None, w.modes_A, w.shape("A"), None,
                                 w.modes_B, w.shape("B"), None, flags)
        if st != 0:
            raise RuntimeError(f"gett_plan: {g.gett_status_string(st)}")
        self.plan = json.loads(g.gett_plan_describe(self.h))

    def launch(self, stream):
        st = self.g.gett_contract(self.h, self.w.alpha, self.A.data_ptr(), self.B.data_ptr(),
                                  self.w.beta, self.C.data_ptr(), stream.cuda_stream)
        if st != 0:
            raise RuntimeError(f"gett_contract: {self.g.gett_status_string(st)}")

    def tune(self, max_candidates: int):
        """gett_plan_tune on this problem's buffers (C is overwritten; it is
        restored from the initial C when beta != 0)."""
        st = self.g.gett_plan_tune(self.h, max_candidates, self.A.data_ptr(), self.B.data_ptr(),
                                   self.C.data_ptr(), 0)
        if st != 0:
            raise RuntimeError(f"gett_plan_tune: {self.g.gett_status_string(st)}")
        if self.C0 is not None:
            self.C.copy_(self.C0)
        self.plan = json.loads(self.g.gett_plan_describe(self.h))

    def close(self):
        self.g.gett_destroy(self.h)


class TtgtProblem:
    """The same workload run by TTGT (Sec. 4): explicit transpositions into a
    workspace, one rocBLAS GEMM, a fold into C."""

    def __init__(self, p: Problem):
        import torch
        g, w = p.g, p.w
        self.p, self.g = p, g
        dt = g.GETT_FLOAT32 if w.dtype == "f32" else g.GETT_FLOAT64
        st, self.h = g.gett_ttgt_plan(dt, w.modes_C, w.shape("C"), None, w.modes_A, w.shape("A"),
                                      None, w.modes_B, w.shape("B"), None, -1)
        if st != 0:
            raise RuntimeError(f"gett_ttgt_plan: {g.gett_status_string(st)}")
        _, self.nws = g.gett_ttgt_workspace_size(self.h)
        self.ws = torch.empty(max(self.nws, 1), dtype=torch.uint8, device=p.dev)
        self.plan = json.loads(g.gett_ttgt_describe(self.h))

    def launch(self, stream):
        p = self.p
        st = self.g.gett_ttgt_contract(self.h, p.w.alpha, p.A.data_ptr(), p.B.data_ptr(), p.w.beta,
                                       p.C.data_ptr(), self.ws.data_ptr(), self.nws,
                                       stream.cuda_stream)
        if st != 0:
            raise RuntimeError(f"gett_ttgt_contract: {self.g.gett_status_string(st)}")

    def close(self):
        self.g.gett_ttgt_destroy(self.h)
        del self.ws


class LogProblem:
    """The same workload run by Loops-over-GEMM (Sec. 5): GEMMs on 2D slices,
    strided-batched over one loop index.  `ok` is False when LoG does not
    apply (Listing 7)."""

    def __init__(self, p: Problem):
        g, w = p.g, p.w
        self.p, self.g = p, g
        dt = g.GETT_FLOAT32 if w.dtype == "f32" else g.GETT_FLOAT64
        st, self.h = g.gett_log_plan(dt, w.modes_C, w.shape("C"), None, w.modes_A, w.shape("A"),
                                     None, w.modes_B, w.shape("B"), None)
        self.ok = st == 0
        if st not in (0, g.GETT_ERROR_NOT_SUPPORTED):
            raise RuntimeError(f"gett_log_plan: {g.gett_status_string(st)}")
        self.plan = json.loads(g.gett_log_describe(self.h)) if self.ok else None

    def launch(self, stream):
        p = self.p
        st = self.g.gett_log_contract(self.h, p.w.alpha, p.A.data_ptr(), p.B.data_ptr(), p.w.beta,
                                      p.C.data_ptr(), stream.cuda_stream)
        if st != 0:
            raise RuntimeError(f"gett_log_contract: {self.g.gett_status_string(st)}")

    def close(self):
        if self.ok:
            self.g.gett_log_destroy(self.h)


class SelectProblem:
    """The same workload run through method selection (Sec. 6): the library
    times GETT, TTGT and LoG on the problem's buffers and keeps the fastest."""

    def __init__(self, p: Problem, stream, max_candidates):
        import torch
        g, w = p.g, p.w
        self.p, self.g = p, g
        dt = g.GETT_FLOAT32 if w.dtype == "f32" else g.GETT_FLOAT64
        st, self.h = g.gett_select_plan(dt, w.modes_C, w.shape("C"), None, w.modes_A,
                                        w.shape("A"), None, w.modes_B, w.shape("B"), None, 0, -1)
        if st != 0:
            raise RuntimeError(f"gett_select_plan: {g.gett_status_string(st)}")
        _, self.nws = g.gett_select_workspace_size(self.h)
        self.ws = torch.empty(max(self.nws, 1), dtype=torch.uint8, device=p.dev)
        scratch = torch.empty_like(p.C)
        st = g.gett_select_tune(self.h, max_candidates, p.A.data_ptr(), p.B.data_ptr(),
                                scratch.data_ptr(), self.ws.data_ptr(), self.nws,
                                stream.cuda_stream)
        del scratch
        if st != 0:
            raise RuntimeError(f"gett_select_tune: {g.gett_status_string(st)}")
        self.plan = json.loads(g.gett_select_describe(self.h))

    def launch(self, stream):
        p = self.p
        st = self.g.gett_select_contract(self.h, p.w.alpha, p.A.data_ptr(), p.B.data_ptr(),
                                         p.w.beta, p.C.data_ptr(), self.ws.data_ptr(), self.nws,
                                         stream.cuda_stream)
        if st != 0:
            raise RuntimeError(f"gett_select_contract: {self.g.gett_status_string(st)}")

    def close(self):
        self.g.gett_select_destroy(self.h)
        del self.ws


def time_log(p: Problem, stream, runs, flush):
    """Cold minimum (ms) of the LoG run of a problem, or None when LoG does not apply."""
    lp = LogProblem(p)
    if not lp.ok:
        return None, None
    for _ in range(2):
        lp.launch(stream)
    t = min(time_launches(lambda: lp.launch(stream), runs, stream, flush))
    calls = lp.plan["gemm_calls"]
    lp.close()
    return t, calls


def cache_flush(dev):
    """Evict the caches between cold runs by reading a 1 GiB buffer (summed
    into a preallocated scalar).  Reading rather than writing leaves no dirty
    lines whose write-back the next kernel would pay for: a write flush adds
    7-11% to the write-only 6D workload's median and 4% to the headline's,
    nothing to compute-bound ones."""
    import torch
    buf = torch.zeros(1 << 28, dtype=torch.float32, device=dev)   # 1 GiB
    sink = torch.empty((), dtype=torch.float32, device=dev)
    return lambda: torch.sum(buf, 0, out=sink)


def time_launches(fn, n, stream, flush=None):
    """Per-launch HIP event times (ms) on `stream`, optionally after a flush."""
    import torch
    ts = []
    for _ in range(n):
        if flush is not None:
            flush()
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        fn()
        e1.record(stream)
        e1.synchronize()
        ts.append(e0.elapsed_time(e1))
    return ts


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, whole_runs=0, target_s=5.0, single_s=0.0):
    """The oracle (plain C, fp64, all host threads) timed on the host.

    whole_runs > 0: all of C, that many runs, the minimum reported (Sec. 7's
    statistic); otherwise one run over an evenly spaced sample of C's
    elements sized to about target_s seconds.  single_s > 0: also one thread
    on a sample of about that many seconds (the paper's numbers are
    single-core)."""
    import oracle
    A, B, Cin = wl.make_inputs(w)
    nC = w.numel("C")
    flops_per_elem = wl.flop_count(w) / nC
    threads = oracle.max_threads()

    def run(n, nthreads):
        pts = np.linspace(0, nC - 1, n).astype(np.int64)
        t = time.perf_counter()
        oracle.contract(w.modes_C, w.modes_A, w.modes_B, A, B, w.alpha, w.beta, Cin,
                        shape_C=w.shape("C"), points=pts, nthreads=nthreads)
        return time.perf_counter() - t

    def sized(nthreads, seconds):
        n0 = min(nC, 50_000)
        dt0 = run(n0, nthreads)
        return int(min(nC, max(n0, n0 * seconds / max(dt0, 1e-6))))

    if whole_runs > 0:
        times = [run(nC, threads) for _ in range(whole_runs)]
        n, dt = nC, min(times)
        sample = (f"all {nC} elements of C ({w.name}), minimum of {whole_runs} runs: "
                  + ", ".join(f"{t:.2f}" for t in times) + " s")
    else:
        n = sized(threads, target_s)
        dt = run(n, threads)
        sample = f"{n} of {nC} elements of C ({w.name}), evenly spaced, one run: {dt:.1f} s"
    rec = {"value": round(flops_per_elem * n / dt / 1e9, 4), "unit": "GFLOP/s", "cores": threads,
           "kind": "oracle", "sample": sample, "cpu_model": cpu_model()}
    if single_s > 0:
        n1 = sized(1, single_s)
        dt1 = run(n1, 1)
        reps = 1
        if n1 == nC and dt1 < single_s / 3:   # all of C is quick: repeat, keep the minimum
            reps = int(min(50, single_s / max(dt1, 1e-6)))
            dt1 = min([dt1] + [run(n1, 1) for _ in range(reps - 1)])
        rec["single_thread_value"] = round(flops_per_elem * n1 / dt1 / 1e9, 4)
        rec["single_thread_sample"] = (f"{n1} of {nC} elements, evenly spaced, one thread: "
                                       f"{dt1:.3f} s" + (f" (minimum of {reps} runs)" if reps > 1 else ""))
    return rec


# Oracle timing per workload: the two small ones over all of C (minimum of
# three runs) and on one core too; the large ones on one bounded sample.
CPU_PLAN = {"tm3x2_fp32": dict(whole_runs=3, single_s=3.0),
            "bw4x3_fp32": dict(whole_runs=3, single_s=3.0),
            "cc4x4_fp64": dict(target_s=5.0), "ccsdt6_fp64": dict(target_s=5.0),
            "gemm4_fp32": dict(target_s=5.0)}


def traffic_for(kernel_name: str, workload: str):
    """HBM bytes per launch from the committed rocprofv3 --pmc summary, or None
    when it was measured on other kernel sources."""
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.json")
    if not os.path.exists(path):
        return None
    try:
        d = json.load(open(path))
    except Exception:
        return None
    if d.get("source_hash") != kernel_source_hash():
        return None
    return d.get("bytes_per_launch")


def roofline_of(w, kernel_ms):
    """The workload's bound (HBM or MFMA), its algorithmic bytes or flops per
    launch over the kernel's average launch time, and the peak."""
    if bound_of(w) == "hbm":
        per = wl.algorithmic_bytes(w)
        roof = {"bound": "hbm", "achieved": round(per / (kernel_ms * 1e-3) / 1e9, 1),
                "peak": PEAK["hbm_GBs"], "unit": "GB/s"}
    else:
        per = wl.flop_count(w)
        pk = PEAK["f32_TFLOPs"] if w.dtype == "f32" else PEAK["f64_TFLOPs"]
        roof = {"bound": "mfma", "achieved": round(per / (kernel_ms * 1e-3) / 1e12, 2),
                "peak": pk, "unit": "TFLOP/s"}
    roof["frac"] = round(roof["achieved"] / roof["peak"], 4)
    roof["traffic"] = traffic_for("gett_macro_kernel", w.name)
    roof["kernel_ms_avg"] = round(kernel_ms, 5)
    return roof


def report_workload(w, dev, stream, runs, flush):
    import torch

    import paper_1607_00145_amd as g
    p = Problem(w, dev)
    flops = wl.flop_count(w)
    nbytes = wl.algorithmic_bytes(w)
    for _ in range(3):
        p.launch(stream)
    ts = time_launches(lambda: p.launch(stream), runs, stream, flush)
    tmin, tmed = min(ts), statistics.median(ts)
    # warm launches back to back: the kernel's average launch time (HIP events)
    warm = time_launches(lambda: p.launch(stream), 50, stream)
    bound = bound_of(w)
    peak_f = (PEAK["f32_TFLOPs"] if w.dtype == "f32" else PEAK["f64_TFLOPs"]) * 1e12
    rec = {"workload": w.name, "expression": w.expression(), "dtype": w.dtype,
           "bound": bound, "ms_min": round(tmin, 5), "ms_median": round(tmed, 5),
           "gflops": round(flops / (tmin * 1e-3) / 1e9, 1),
           "gbs": round(nbytes / (tmin * 1e-3) / 1e9, 1)}
    rec["frac_mfma_peak"] = round(flops / (tmin * 1e-3) / peak_f, 4)
    rec["frac_hbm_peak"] = round(nbytes / (tmin * 1e-3) / (PEAK["hbm_GBs"] * 1e9), 4)
    rec["frac_of_bound"] = rec["frac_mfma_peak"] if bound == "mfma" else rec["frac_hbm_peak"]
    rec["plan"] = {k: p.plan[k] for k in ("swapped", "merges", "x_order", "y_order", "k_order",
                                           "gather_x", "gather_y", "c_vector")}
    rec["plan"]["tile"] = [p.plan["tile"]["mt"], p.plan["tile"]["nt"], p.plan["tile"]["kt"]]
    rec["plan"]["workgroups"] = p.plan["grid"]["workgroups"]
    rec["plan"]["kslices"] = p.plan["kslices"]
    rec["plan"]["kernel"] = p.plan["kernel"]
    rec["plan"]["partials"] = p.plan["partials"]
    if p.plan["kernel"] == "tail":
        rec["plan"]["tail"] = p.plan["tail"]
    rec["roofline"] = roofline_of(w, statistics.mean(warm))
    # results are identical from call to call in every plan (partial tiles are
    # summed in a fixed order); where the plan has partial tiles, the same
    # contraction in whole tiles only is timed beside it
    rec["deterministic"] = True
    if p.plan["partials"] != "none":
        pw = Problem(w, dev, flags=g.GETT_FLAG_WHOLE_TILES)
        for _ in range(3):
            pw.launch(stream)
        tw = time_launches(lambda: pw.launch(stream), runs, stream, flush)
        rec["whole_tiles_ms_min"] = round(min(tw), 5)
        rec["whole_tiles_ms_median"] = round(statistics.median(tw), 5)
        pw.close()
        del pw
    t = TtgtProblem(p)
    for _ in range(3):
        t.launch(stream)
    tt = min(time_launches(lambda: t.launch(stream), runs, stream, flush))
    rec["ttgt_ms_min"] = round(tt, 5)
    rec["ttgt_gflops"] = round(flops / (tt * 1e-3) / 1e9, 1)
    rec["ttgt_transposed"] = t.plan["transposed"]
    rec["ttgt_workspace_bytes"] = t.plan["workspace_bytes"]
    rec["gett_speedup_over_ttgt"] = round(tt / tmin, 3)
    t.close()
    tl, calls = time_log(p, stream, runs, flush)
    rec["log_ms_min"] = round(tl, 5) if tl else None
    rec["log_gemm_calls"] = calls
    rec["gett_speedup_over_log"] = round(tl / tmin, 3) if tl else None
    p.close()
    M, N, K = p.plan["size_x"], p.plan["size_y"], p.plan["size_k"]
    del p
    gmin = time_gemm(M, N, K, w, dev, stream, runs, flush)
    rec["gemm_ms_min"] = round(gmin, 5)
    rec["gemm_gflops"] = round(flops / (gmin * 1e-3) / 1e9, 1)
    rec["vs_equal_size_gemm"] = round(gmin / tmin, 4)
    return rec


def time_gemm(M, N, K, w, dev, stream, runs, flush):
    """Cold minimum (ms) of the equal-size GEMM of Sec. 7 (S_Im x S_Ik times
    S_Ik x S_In with the workload's alpha and beta) through torch."""
    import torch
    torch.cuda.empty_cache()
    dt = torch.float32 if w.dtype == "f32" else torch.float64
    torch.backends.cuda.matmul.allow_tf32 = False
    a = torch.randn(M, K, dtype=dt, device=dev)
    b = torch.randn(K, N, dtype=dt, device=dev)
    c = torch.randn(M, N, dtype=dt, device=dev)
    if w.beta != 0:
        fn = lambda: torch.addmm(c, a, b, beta=w.beta, alpha=w.alpha, out=c)
    else:
        fn = lambda: torch.mm(a, b, out=c)
    for _ in range(3):
        fn()
    gmin = min(time_launches(fn, runs, stream, flush))
    del a, b, c
    torch.cuda.empty_cache()
    return gmin


TRANSPOSE_CASES = [   # (name, dtype, extents, perm): Eq. 4 with alpha 1, beta 0
    ("t4_rev_fp32", "f32", [112, 112, 112, 112], [3, 2, 1, 0]),
    ("t4_keep_fp32", "f32", [112, 112, 112, 112], [0, 2, 3, 1]),
    ("t6_rev_fp64", "f64", [24] * 6, [5, 4, 3, 2, 1, 0]),
    ("t2_fp32", "f32", [8192, 8192], [1, 0]),
]


def report_transpose(dev, stream, runs, flush):
    """The Eq. 4 kernel alone: bytes read + written per launch over its cold time."""
    import torch

    import paper_1607_00145_amd as g
    out = []
    for name, dtype, ext, perm in TRANSPOSE_CASES:
        tdt = torch.float32 if dtype == "f32" else torch.float64
        n = int(np.prod(ext))
        src = torch.rand(n, dtype=tdt, device=dev)
        dst = torch.empty(n, dtype=tdt, device=dev)
        sin = list(np.cumprod([1] + ext[:-1]))
        oext = [ext[p] for p in perm]
        ostr = list(np.cumprod([1] + oext[:-1]))
        sout = [0] * len(ext)
        for j, d in enumerate(perm):
            sout[d] = int(ostr[j])
        code = g.GETT_FLOAT32 if dtype == "f32" else g.GETT_FLOAT64

        def fn():
            st = g.gett_transpose(code, ext, sin, sout, 1.0, src.data_ptr(), 0.0, dst.data_ptr(),
                                  stream.cuda_stream)
            if st != 0:
                raise RuntimeError(g.gett_status_string(st))
        for _ in range(3):
            fn()
        t = min(time_launches(fn, runs, stream, flush))
        nbytes = 2 * n * src.element_size()
        out.append({"case": name, "extents": ext, "perm": perm, "ms_min": round(t, 5),
                    "gbs": round(nbytes / (t * 1e-3) / 1e9, 1),
                    "frac_hbm_peak": round(nbytes / (t * 1e-3) / (PEAK["hbm_GBs"] * 1e9), 4)})
        del src, dst
        torch.cuda.empty_cache()
    return out


def sweep_points(sweep):
    """(tag, workload) pairs of a sweep: Fig. 11 (Sec. 7.3) or the benchmark
    of Appendix A (Tables III / IV)."""
    if sweep == "fig11":
        for dtype in ("f32", "f64"):
            for variant in ("a", "b"):
                for k in wl.FIG11_K:
                    yield "fig11", wl.fig11(variant, k, dtype)
    else:
        from workloads.appendix_a import appendix_workloads
        for dtype in ("f32", "f64"):
            for w in appendix_workloads(dtype):
                yield "appendix_a", w


def sweep_run(sweep, dev, stream, runs, flush, max_candidates):
    """One JSON line per point: GETT with the model's choice, GETT after
    gett_plan_tune over the best `max_candidates` candidates, TTGT, LoG (when
    it applies) and the equal-size GEMM, all cold."""
    for tag, w in sweep_points(sweep):
        dtype = w.dtype
        peak = (PEAK["f32_TFLOPs"] if dtype == "f32" else PEAK["f64_TFLOPs"]) * 1e12
        k = w.extents.get("k")
        flops = wl.flop_count(w)
        p = Problem(w, dev, on_device=True)
        tile = lambda: [p.plan["tile"][x] for x in ("mt", "nt", "kt")] + [
            p.plan["kernel"] if p.plan["kslices"] == 1 else f"kslices{p.plan['kslices']}"]
        model_tile = tile()
        for _ in range(3):
            p.launch(stream)
        tm = min(time_launches(lambda: p.launch(stream), runs, stream, flush))
        p.tune(max_candidates)
        for _ in range(3):
            p.launch(stream)
        tt = min(time_launches(lambda: p.launch(stream), runs, stream, flush))
        tuned_tile = tile()
        M, N, K = p.plan["size_x"], p.plan["size_y"], p.plan["size_k"]
        t = TtgtProblem(p)
        for _ in range(3):
            t.launch(stream)
        tx = min(time_launches(lambda: t.launch(stream), runs, stream, flush))
        t.close()
        tl, _ = time_log(p, stream, runs, flush)
        # method selection: its GETT plan starts from the tuned choice above
        sp = SelectProblem(p, stream, 0)
        for _ in range(2):
            sp.launch(stream)
        ts = min(time_launches(lambda: sp.launch(stream), runs, stream, flush))
        smethod = sp.plan["method"]
        sp.close()
        p.close()
        del p
        tg = time_gemm(M, N, K, w, dev, stream, runs, flush)
        best = min(tm, tt)
        rec = {"sweep": tag, "contraction": w.name, "expression": w.expression(),
               "dtype": dtype, "S_Ik": k if tag == "fig11" else None, "bound": bound_of(w),
               "model_ms": round(tm, 5), "model_tile": model_tile,
               "model_gflops": round(flops / (tm * 1e-3) / 1e9, 1),
               "tuned_ms": round(tt, 5), "tuned_tile": tuned_tile,
               "tuned_gflops": round(flops / (tt * 1e-3) / 1e9, 1),
               "model_of_best": round(best / tm, 4),
               "frac_mfma_peak": round(flops / (best * 1e-3) / peak, 4),
               "frac_hbm_peak": round(wl.algorithmic_bytes(w) / (best * 1e-3) /
                                      (PEAK["hbm_GBs"] * 1e9), 4),
               "ttgt_ms": round(tx, 5), "ttgt_gflops": round(flops / (tx * 1e-3) / 1e9, 1),
               "log_ms": round(tl, 5) if tl else None,
               "log_gflops": round(flops / (tl * 1e-3) / 1e9, 1) if tl else None,
               "gemm_ms": round(tg, 5),
               "gemm_gflops": round(flops / (tg * 1e-3) / 1e9, 1),
               "vs_equal_size_gemm": round(tg / best, 4),
               "select_method": smethod, "select_ms": round(ts, 5),
               "select_vs_equal_size_gemm": round(tg / ts, 4)}
        log(f"[sweep] {w.name}: model {tm*1e3:.1f} us, tuned {tt*1e3:.1f} us, "
            f"ttgt {tx*1e3:.1f} us, log {tl*1e3 if tl else float('nan'):.1f} us, "
            f"gemm {tg*1e3:.1f} us")
        print(json.dumps(rec), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default=HEADLINE, choices=[w.name for w in wl.WORKLOADS])
    ap.add_argument("--report-runs", type=int, default=20)
    ap.add_argument("--no-report", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--sweep", choices=["fig11", "appendix_a"], default=None,
                    help="run a sweep instead: the S_Ik sweep of Fig. 11 or the 48-contraction "
                         "benchmark of Appendix A (one JSON line per point)")
    ap.add_argument("--max-candidates", type=int, default=16,
                    help="candidates gett_plan_tune times in the sweep")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB a few times (the reference "
                         "for scaling rocprofv3 FETCH_SIZE / WRITE_SIZE)")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU: the contraction is built and timed on a single "
              "MI355X; --gpus above 1 is not supported", file=sys.stderr)
        sys.exit(2)

    import torch
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    import paper_1607_00145_amd as g
    g.load_library()   # fails loudly when the HIP library is not built
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    if args.calibrate_copy:
        n = args.calibrate_copy * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"calibrate_copy_bytes": n * 4, "launches": 5}), flush=True)
        return
    if args.sweep:
        sweep_run(args.sweep, dev, stream, args.report_runs, cache_flush(dev),
                  args.max_candidates)
        return
    w = wl.BY_NAME[args.workload]

    # ---- headline: K back-to-back steps, inputs resident ----
    p = Problem(w, dev)
    log(f"[bench] {w.name}: plan {json.dumps({k: p.plan[k] for k in ('tile', 'kbox', 'grid')})}")
    for _ in range(args.warmup):
        p.launch(stream)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        p.launch(stream)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    ms_per_step = elapsed / args.steps * 1e3
    flops = wl.flop_count(w)
    value = flops * args.steps / elapsed / 1e9
    # live per-launch kernel time (HIP events on the launch stream)
    ev = time_launches(lambda: p.launch(stream), max(20, min(args.steps, 200)), stream)
    roof = roofline_of(w, statistics.mean(ev))
    p.close()
    del p
    torch.cuda.empty_cache()

    out = {"metric": "GFLOP/s", "value": round(value, 1), "unit": "GFLOP/s", "n_gpus": 1,
           "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms_per_step, 5),
           "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
           "dtype": w.dtype, "data": "synthetic (seeded PCG64, workloads module)",
           "config": {"workload": w.name, "expression": w.expression(),
                      "extents": w.extents, "alpha": w.alpha, "beta": w.beta,
                      "layout": "column-major", "parallelism": "single GPU",
                      "deterministic": True,
                      "headline": "the fp32 bandwidth-bound 4D x 3D contraction is the "
                                  "configuration the metric is quoted on; every workload "
                                  "(the 4096^3-shaped one included) has its own record with "
                                  "roofline and CPU baseline under workloads"},
           "roofline": roof}

    # ---- per-workload cold-cache report ----
    if not args.no_report:
        flush = cache_flush(dev)
        reps = []
        for ww in wl.WORKLOADS:
            log(f"[bench] report {ww.name}")
            reps.append(report_workload(ww, dev, stream, args.report_runs, flush))
        out["workloads"] = reps
        log("[bench] report transpose")
        out["transpose"] = report_transpose(dev, stream, args.report_runs, flush)
        del flush
        torch.cuda.empty_cache()

    if not args.no_cpu_baseline:
        log("[bench] cpu baseline (oracle)")
        out["cpu_baseline"] = cpu_baseline(w, **CPU_PLAN.get(w.name, {}))
        for rec in out.get("workloads", []):
            if rec["workload"] == w.name:
                rec["cpu_baseline"] = out["cpu_baseline"]
                continue
            log(f"[bench] cpu baseline (oracle) {rec['workload']}")
            rec["cpu_baseline"] = cpu_baseline(wl.BY_NAME[rec["workload"]],
                                               **CPU_PLAN.get(rec["workload"], {}))
            rec["vs_cpu_baseline"] = round(rec["gflops"] / rec["cpu_baseline"]["value"], 1)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
