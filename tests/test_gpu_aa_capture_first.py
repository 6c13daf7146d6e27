"""A direct-load kernel's first launch inside a HIP graph capture.

On a kernel's first launch on a device the library raises that kernel's
dynamic LDS cap (hipFuncSetAttribute) and, for the persistent kernel, looks
up how many of its workgroups are resident; gett_contract_noalloc promises
callers under graph capture that no eager call is needed first.  This file is
collected before every other GPU test (by its name), so in a full run these
captures are the kernels' first launches in the process: captured once,
replayed three times with eager work between the replays, every replay
bit-identical to an eager call after them (integer-valued inputs)."""
import json

import numpy as np
import pytest

import paper_1607_00145_amd as g

pytestmark = pytest.mark.gpu

CASES = {
    # (dtype, forced tile, forced kind, kernel in the plan's description, modes, extents)
    "direct_fp32": (np.float32, "8", "4", "direct", ("a,b", "a,k", "k,b"),
                    {"a": 512, "b": 512, "k": 64}),
    "direct_stream_fp64": (np.float64, "14", "5", "direct-stream", ("a,b", "a,k", "k,b"),
                           {"a": 2048, "b": 2560, "k": 24}),
}


@pytest.mark.parametrize("name", list(CASES))
def test_first_launch_captured(gpu, monkeypatch, name):
    import torch
    dtype, tile, kind, kernel, modes, ext = CASES[name]
    monkeypatch.setenv("GETT_FORCE_TILE", tile)
    monkeypatch.setenv("GETT_FORCE_KIND", kind)
    shp = lambda m: [ext[x] for x in m.split(",")]
    code = g.GETT_FLOAT32 if dtype == np.float32 else g.GETT_FLOAT64
    tdt = torch.float32 if dtype == np.float32 else torch.float64
    gen = torch.Generator(device="cpu").manual_seed(5)
    rnd = lambda n: torch.randint(-3, 4, (n,), generator=gen).to(tdt).to(gpu)
    A = rnd(int(np.prod(shp(modes[1]))))
    B = rnd(int(np.prod(shp(modes[2]))))
    nC = int(np.prod(shp(modes[0])))
    st, h = g.gett_plan(code, modes[0], shp(modes[0]), None, modes[1], shp(modes[1]), None,
                        modes[2], shp(modes[2]), None, 0)
    assert st == 0
    try:
        assert json.loads(g.gett_plan_describe(h))["kernel"] == kernel
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        C = torch.full((nC,), float("nan"), dtype=tdt, device=gpu)
        torch.cuda.synchronize()
        graph = torch.cuda.CUDAGraph()
        with torch.cuda.graph(graph, stream=side):
            st = g.gett_contract_noalloc(h, 1.0, A.data_ptr(), B.data_ptr(), 0.0, C.data_ptr(),
                                         side.cuda_stream)
        assert st == 0, g.gett_status_string(st)
        outs = []
        for rep in range(3):
            C.fill_(float("nan"))
            torch.cuda.synchronize()
            graph.replay()
            torch.cuda.synchronize()
            outs.append(C.clone())
            _ = (A * 2).sum().item()   # eager work between the replays
        ref = torch.full((nC,), float("nan"), dtype=tdt, device=gpu)
        assert g.gett_contract(h, 1.0, A.data_ptr(), B.data_ptr(), 0.0, ref.data_ptr(),
                               torch.cuda.current_stream().cuda_stream) == 0
        torch.cuda.synchronize()
        assert bool(torch.isfinite(ref).all())
        for rep, out in enumerate(outs):
            assert torch.equal(out, ref), f"replay {rep} differs from the eager call"
        del graph
    finally:
        g.gett_destroy(h)
