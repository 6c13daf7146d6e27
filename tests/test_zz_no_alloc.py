"""gett_contract_noalloc: the same contraction as gett_contract with the
partial-tile workspace taken from the library's fixed static buffer (for
callers that cannot allocate device memory).  Through the C interface, on
plans with a stream-K tail, with K slices and with whole tiles: two calls in a
row, the second on a smaller contraction, each bit-identical to gett_contract
(the same kernels sum in the same order) and within the parity bar of the
oracle; a plan whose workspace exceeds the buffer is refused before any
launch; a call captured into a HIP graph without any eager call first
replays correctly."""
import json

import numpy as np
import pytest

import paper_1607_00145_amd as g
import workloads as wl
from gpu_util import TOL, compare_whole, split

pytestmark = pytest.mark.gpu
TAIL_TILE = {"f32": "2", "f64": "8"}

# (name, forced choices, larger extents, smaller extents): the second call of
# each pair runs the smaller contraction
PAIRS = [
    ("tail", {"GETT_FORCE_KIND": "3", "GETT_TAIL_WGS": "7"},
     (("a,b", "a,k", "k,b"), {"a": 300, "b": 290, "k": 333}),
     (("a,b", "a,k", "k,b"), {"a": 150, "b": 170, "k": 211})),
    ("kslices", {"GETT_FORCE_KSLICES": "8"},
     (("a,b", "a,c,d", "d,b,c"), {"a": 45, "b": 38, "c": 29, "d": 37}),
     (("a,b", "a,c,d", "d,b,c"), {"a": 21, "b": 30, "c": 17, "d": 13})),
    ("whole", {},
     (("a,b,c,d", "a,e,b", "e,d,c"), {"a": 40, "b": 36, "c": 50, "d": 44, "e": 16}),
     (("a,b,c,d", "a,e,b", "e,d,c"), {"a": 12, "b": 9, "c": 20, "d": 7, "e": 16})),
]


def plan_of(modes, ext, dtype):
    code = g.GETT_FLOAT32 if dtype == "f32" else g.GETT_FLOAT64
    sh = [[ext[x] for x in split(m)] for m in modes]
    st, h = g.gett_plan(code, modes[0], sh[0], None, modes[1], sh[1], None, modes[2], sh[2],
                        None, 0)
    assert st == 0, g.gett_status_string(st)
    return h, json.loads(g.gett_plan_describe(h))


def both(gpu, w, h):
    """C from gett_contract and from gett_contract_noalloc on the same inputs."""
    import torch
    A, B, Cin = wl.make_inputs(w)
    flat = lambda t: torch.from_numpy(np.asfortranarray(t).reshape(-1, order="F")).to(gpu)
    tA, tB = flat(A), flat(B)
    C0 = flat(Cin) if Cin is not None else torch.full((w.numel("C"),), float("nan"),
                                                         dtype=tA.dtype, device=gpu)
    s = torch.cuda.current_stream().cuda_stream
    ref, got = C0.clone(), C0.clone()
    assert g.gett_contract(h, w.alpha, tA.data_ptr(), tB.data_ptr(), w.beta, ref.data_ptr(), s) == 0
    assert g.gett_contract_noalloc(h, w.alpha, tA.data_ptr(), tB.data_ptr(), w.beta,
                                   got.data_ptr(), s) == 0
    torch.cuda.synchronize()
    return (A, B, Cin), ref, got


@pytest.mark.parametrize("dtype", ["f32", "f64"])
@pytest.mark.parametrize("case", range(len(PAIRS)), ids=[p[0] for p in PAIRS])
def test_noalloc_matches_contract_two_calls(gpu, monkeypatch, case, dtype):
    import torch
    name, env, big, small = PAIRS[case]
    for k, v in env.items():
        monkeypatch.setenv(k, v)
    if name == "tail":
        monkeypatch.setenv("GETT_FORCE_TILE", TAIL_TILE[dtype])
    for n, (modes, ext) in enumerate((big, small)):
        w = wl.Workload(880 + 10 * case + n, f"{name}{n}", dtype, *modes, ext, alpha=-1.25,
                        beta=0.5 if n else 0.0)
        h, d = plan_of(modes, ext, dtype)
        try:
            if name == "tail":
                assert d["kernel"] == "tail"
            if name == "kslices":
                assert d["kslices"] == 8
            if name != "whole":
                assert d["partials"] == "workspace" and d["workspace_bytes"] > 0
            host, ref, got = both(gpu, w, h)
            assert torch.equal(ref, got), f"call {n}: noalloc differs from gett_contract"
            assert compare_whole(got, w, *host) <= TOL[w.np_dtype]
        finally:
            g.gett_destroy(h)


def test_noalloc_full_size_tail_then_smaller(gpu):
    """The model's plan for the 4D x 4D fp64 workload (stream-K tail, about
    25 MB of partial tiles), then a smaller contraction of the same form."""
    import torch
    w = wl.WORKLOADS[2]
    small = wl.scaled(w, {"a": 40, "b": 36, "i": 44, "j": 30, "e": 20, "f": 50})
    for ww in (w, small):
        h, d = plan_of((ww.modes_C, ww.modes_A, ww.modes_B), ww.extents, "f64")
        try:
            host, ref, got = both(gpu, ww, h)
            assert torch.equal(ref, got), ww.name
            assert compare_whole(got, ww, *host) <= TOL[np.float64]
        finally:
            g.gett_destroy(h)


def test_noalloc_refuses_a_workspace_beyond_the_buffer(gpu, monkeypatch):
    """256 slices of 256 tiles of 128 x 128 fp32 need 4 GiB of partial tiles:
    refused (GETT_ERROR_NOT_SUPPORTED) before any launch, C untouched."""
    import torch
    monkeypatch.setenv("GETT_FORCE_KSLICES", "256")
    monkeypatch.setenv("GETT_FORCE_TILE", "0")
    ext = {"a": 2048, "b": 2048, "k": 4096}
    h, d = plan_of(("a,b", "a,k", "k,b"), ext, "f32")
    try:
        assert d["kslices"] == 256 and d["workspace_bytes"] > (64 << 20)
        A = torch.zeros(2048 * 4096, device=gpu)
        B = torch.zeros(4096 * 2048, device=gpu)
        C = torch.full((2048 * 2048,), 7.0, device=gpu)
        st = g.gett_contract_noalloc(h, 1.0, A.data_ptr(), B.data_ptr(), 0.0, C.data_ptr(),
                                     torch.cuda.current_stream().cuda_stream)
        assert st == g.GETT_ERROR_NOT_SUPPORTED
        torch.cuda.synchronize()
        assert bool((C == 7.0).all()), "a refused call must not touch C"
    finally:
        g.gett_destroy(h)


def test_noalloc_under_graph_capture(gpu, monkeypatch):
    """Captured with no eager call before (nothing to allocate), replayed four
    times with eager work between the replays: every replay equals the eager
    gett_contract result bit for bit."""
    import torch
    monkeypatch.setenv("GETT_FORCE_KSLICES", "8")
    w = wl.Workload(899, "graph", "f64", "a,b", "a,k", "k,b", {"a": 200, "b": 180, "k": 900},
                    alpha=1.5, beta=-0.5)
    A, B, Cin = wl.make_inputs(w)
    flat = lambda t: torch.from_numpy(np.asfortranarray(t).reshape(-1, order="F")).to(gpu)
    tA, tB, C0 = flat(A), flat(B), flat(Cin)
    h, d = plan_of(("a,b", "a,k", "k,b"), w.extents, "f64")
    try:
        assert d["kslices"] == 8
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        Cg = C0.clone()
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.stream(side):
            with torch.cuda.graph(graph, stream=side):
                st = g.gett_contract_noalloc(h, w.alpha, tA.data_ptr(), tB.data_ptr(), w.beta,
                                             Cg.data_ptr(), side.cuda_stream)
        assert st == 0
        torch.cuda.synchronize()
        ref = C0.clone()
        assert g.gett_contract(h, w.alpha, tA.data_ptr(), tB.data_ptr(), w.beta, ref.data_ptr(),
                               torch.cuda.current_stream().cuda_stream) == 0
        torch.cuda.synchronize()
        for rep in range(4):
            Cg.copy_(C0)
            junk = (tA * 2).sum()
            torch.cuda.synchronize()
            graph.replay()
            torch.cuda.synchronize()
            assert torch.equal(Cg, ref), f"replay {rep}"
            del junk
        assert compare_whole(ref, w, A, B, Cin) <= TOL[np.float64]
    finally:
        g.gett_destroy(h)
