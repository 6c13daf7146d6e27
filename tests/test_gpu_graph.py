"""gett_contract under HIP graph capture (serving loops replay one captured
contraction): a plain plan, plans over K slices and with a stream-K tail
(partial tiles summed through the library's workspace), the direct-load
kernels and an alpha = 0 call, each captured once and replayed several
times with eager work between the replays; every replay must equal the eager result bit for
bit (integer-valued inputs make every sum exact).  The eager call runs
on the capture stream first: it allocates the stream's workspace, which a
capture must not do."""
import json

import numpy as np
import pytest

import paper_1607_00145_amd as g

pytestmark = pytest.mark.gpu

CASES = {
    # (modes C, A, B), extents, environment of the plan (forced choices)
    "plain": (("a,b,c,d", "a,e,b", "e,d,c"), {"a": 40, "b": 36, "c": 50, "d": 44, "e": 16}, {}),
    "kslices": (("a,b", "a,c,d", "d,b,c"), {"a": 96, "b": 94, "c": 94, "d": 96}, {}),
    "kslices_forced": (("a,b,c", "a,k,c", "k,b"), {"a": 33, "b": 47, "c": 5, "k": 600},
                       {"GETT_FORCE_KSLICES": "8"}),
    "tail_forced": (("a,b", "a,k", "k,b"), {"a": 300, "b": 290, "k": 333},
                    {"GETT_FORCE_KIND": "3", "GETT_TAIL_WGS": "5"}),
    # the direct-load kernel (fp32 only; fp64 runs the tile's macro-kernel):
    # dynamic LDS, loads straight into LDS, ragged tiles and a partial box
    "direct_forced": (("a,b", "a,k", "k,b"), {"a": 300, "b": 260, "k": 104},
                      {"GETT_FORCE_TILE": "8", "GETT_FORCE_KIND": "4"}),
    # the persistent direct-load kernel (fp64 only): workgroups that walk
    # several tiles, a partial K box
    "direct_stream_forced": (("a,b", "a,k", "k,b"), {"a": 2000, "b": 2600, "k": 22},
                             {"GETT_FORCE_TILE": "14", "GETT_FORCE_KIND": "5"}),
}
TAIL_TILE = {np.float32: "2", np.float64: "8"}


@pytest.mark.parametrize("dtype", [np.float32, np.float64])
@pytest.mark.parametrize("alpha,beta", [(1.0, 0.0), (2.0, -1.0), (0.0, 3.0)])
@pytest.mark.parametrize("name", list(CASES))
def test_graph_replay_matches_eager(gpu, monkeypatch, name, alpha, beta, dtype):
    import torch
    modes, ext, env = CASES[name]
    for k, v in env.items():
        monkeypatch.setenv(k, v)
    if name.startswith("tail"):
        monkeypatch.setenv("GETT_FORCE_TILE", TAIL_TILE[dtype])
    sp = lambda m: m.split(",")
    shp = lambda m: [ext[x] for x in sp(m)]
    tdt = torch.float32 if dtype == np.float32 else torch.float64
    code = g.GETT_FLOAT32 if dtype == np.float32 else g.GETT_FLOAT64
    gen = torch.Generator(device="cpu").manual_seed(11)
    rnd = lambda n: torch.randint(-4, 5, (n,), generator=gen).to(tdt).to(gpu)
    nA = int(np.prod(shp(modes[1])))
    nB = int(np.prod(shp(modes[2])))
    nC = int(np.prod(shp(modes[0])))
    A, B, C0 = rnd(nA), rnd(nB), rnd(nC)
    flags = 0
    st, h = g.gett_plan(code, modes[0], shp(modes[0]), None, modes[1], shp(modes[1]), None,
                        modes[2], shp(modes[2]), None, flags)
    assert st == 0
    try:
        d = json.loads(g.gett_plan_describe(h))
        if name.startswith("kslices"):
            assert d["kslices"] > 1
        if name.startswith("tail"):
            assert d["kernel"] == "tail" and d["tail"]["full_tiles"] > 0
        if name.startswith("direct_forced") and dtype == np.float32:
            assert d["kernel"] == "direct"
        if name.startswith("direct_stream") and dtype == np.float64:
            assert d["kernel"] == "direct-stream"
        if d["kslices"] > 1 or d["kernel"] == "tail":
            assert d["partials"] == "workspace"
        # eager reference, on the stream that captures
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        C = C0.clone()
        torch.cuda.synchronize()
        assert g.gett_contract(h, alpha, A.data_ptr(), B.data_ptr(), beta, C.data_ptr(),
                               side.cuda_stream) == 0
        torch.cuda.synchronize()
        ref = C.clone()
        # capture once
        Cg = C0.clone()
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.stream(side):
            with torch.cuda.graph(graph, stream=side):
                st = g.gett_contract(h, alpha, A.data_ptr(), B.data_ptr(), beta, Cg.data_ptr(),
                                     side.cuda_stream)
        assert st == 0
        torch.cuda.synchronize()
        for rep in range(4):
            Cg.copy_(C0)                      # eager work between replays
            junk = (A * 2).sum()              # unrelated eager kernels
            torch.cuda.synchronize()
            graph.replay()
            torch.cuda.synchronize()
            assert torch.equal(Cg, ref), f"replay {rep}"
            del junk
    finally:
        g.gett_destroy(h)


def test_first_call_under_capture_is_refused(gpu, monkeypatch):
    """A plan with partial tiles whose stream has no workspace yet: called
    during a capture it is refused (GETT_ERROR_NOT_SUPPORTED) with nothing
    enqueued -- the workspace would have to be allocated inside the capture.
    The capture itself stays valid, and the same call made eagerly afterwards
    allocates the workspace and computes C."""
    import torch
    monkeypatch.setenv("GETT_FORCE_KSLICES", "8")
    modes, ext, _ = CASES["kslices_forced"]
    shp = lambda m: [ext[x] for x in m.split(",")]
    st, h = g.gett_plan(g.GETT_FLOAT64, modes[0], shp(modes[0]), None, modes[1], shp(modes[1]),
                        None, modes[2], shp(modes[2]), None, 0)
    assert st == 0
    try:
        assert json.loads(g.gett_plan_describe(h))["partials"] == "workspace"
        n = lambda m: int(np.prod(shp(m)))
        A = torch.ones(n(modes[1]), dtype=torch.float64, device=gpu)
        B = torch.ones(n(modes[2]), dtype=torch.float64, device=gpu)
        C = torch.full((n(modes[0]),), 7.0, dtype=torch.float64, device=gpu)
        side = torch.cuda.Stream()                      # a stream never used by the library
        side.wait_stream(torch.cuda.current_stream())
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.stream(side):
            with torch.cuda.graph(graph, stream=side):
                C.mul_(1.0)                             # keep the graph non-empty
                st = g.gett_contract(h, 1.0, A.data_ptr(), B.data_ptr(), 0.0, C.data_ptr(),
                                     side.cuda_stream)
        assert st == g.GETT_ERROR_NOT_SUPPORTED
        graph.replay()
        torch.cuda.synchronize()
        assert torch.all(C == 7.0)                      # the contraction was not captured
        assert g.gett_contract(h, 1.0, A.data_ptr(), B.data_ptr(), 0.0, C.data_ptr(),
                               side.cuda_stream) == 0
        torch.cuda.synchronize()
        assert torch.all(C == float(ext["k"]))          # sum over k of 1 * 1
    finally:
        g.gett_destroy(h)
