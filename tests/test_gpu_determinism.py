"""Results identical from call to call.  Listing 4 sums each tile's contracted
loop in one order; the library keeps a fixed order for the partial tiles of K
slices and of the stream-K tail too (saved to its workspace and summed in
piece order by the last piece of each tile to finish).  Repeated calls on the
same non-integer inputs must give bit-identical C: for the plan the model
makes for the full-size 4D x 4D fp64 workload (a stream-K tail) and for forced
K slices and tails.  Also: one stream's workspace serves plans of different
sizes in turn; two streams run one plan at once; a C in host memory works
(the kernels write C with plain stores only: no atomics touch caller
memory)."""
import json

import numpy as np
import pytest

import paper_1607_00145_amd as g
import workloads as wl
from gpu_util import TOL, compare_whole, split

pytestmark = pytest.mark.gpu
TAIL_TILE = {np.float32: "2", np.float64: "8"}


def plan(modes, ext, dtype, flags=0):
    code = g.GETT_FLOAT32 if dtype == np.float32 else g.GETT_FLOAT64
    sh = [[ext[x] for x in split(m)] for m in modes]
    st, h = g.gett_plan(code, modes[0], sh[0], None, modes[1], sh[1], None, modes[2], sh[2],
                        None, flags)
    assert st == 0, g.gett_status_string(st)
    return h, json.loads(g.gett_plan_describe(h))


def device_inputs(gpu, w):
    import torch
    A, B, Cin = wl.make_inputs(w)
    flat = lambda t: torch.from_numpy(np.asfortranarray(t).reshape(-1, order="F")).to(gpu)
    C0 = flat(Cin) if Cin is not None else torch.zeros(w.numel("C"), dtype=flat(A).dtype,
                                                         device=gpu)
    return (A, B, Cin), flat(A), flat(B), C0


def run(h, w, tA, tB, C, stream=None):
    import torch
    s = stream if stream is not None else torch.cuda.current_stream()
    st = g.gett_contract(h, w.alpha, tA.data_ptr(), tB.data_ptr(), w.beta, C.data_ptr(),
                         s.cuda_stream)
    assert st == 0, g.gett_status_string(st)


def test_full_size_cc4x4_repeatable(gpu):
    """The model's plan for C[a,b,i,j] = A[i,e,j,f] B[f,a,e,b] (all 48, fp64,
    N(0,1) operands): a stream-K tail whose pieces go through the workspace.
    Five calls, five bit-identical results, matching the oracle."""
    import torch
    w = wl.WORKLOADS[2]
    host, tA, tB, C0 = device_inputs(gpu, w)
    h, d = plan((w.modes_C, w.modes_A, w.modes_B), w.extents, np.float64)
    try:
        assert d["kernel"] == "tail" and d["partials"] == "workspace"
        outs = []
        for _ in range(5):
            C = C0.clone()
            run(h, w, tA, tB, C)
            torch.cuda.synchronize()
            outs.append(C)
        for k in range(1, 5):
            assert torch.equal(outs[0], outs[k]), f"call {k} differs from call 0"
        err = compare_whole(outs[0], w, *host)
        assert err <= TOL[np.float64], f"rel err {err:.3e}"
    finally:
        g.gett_destroy(h)


FORCED = [
    ("kslices8", (("a,b", "a,c,d", "d,b,c"), {"a": 45, "b": 38, "c": 29, "d": 37}),
     {"GETT_FORCE_KSLICES": "8"}),
    ("kslices64", (("a,b", "a,k", "k,b"), {"a": 33, "b": 70, "k": 1000}),
     {"GETT_FORCE_KSLICES": "64"}),
    ("tail7", (("a,b", "a,k", "k,b"), {"a": 300, "b": 290, "k": 333}),
     {"GETT_FORCE_KIND": "3", "GETT_TAIL_WGS": "7"}),
    ("tail256", (("a,b,i,j", "i,e,j,f", "f,a,e,b"),
                 {"a": 23, "b": 17, "i": 19, "j": 21, "e": 13, "f": 11}),
     {"GETT_FORCE_KIND": "3", "GETT_TAIL_WGS": "256"}),
]


@pytest.mark.parametrize("dtype", [np.float32, np.float64])
@pytest.mark.parametrize("case", range(len(FORCED)), ids=[c[0] for c in FORCED])
def test_forced_partials_repeatable(gpu, monkeypatch, case, dtype):
    import torch
    name, (modes, ext), env = FORCED[case]
    for k, v in env.items():
        monkeypatch.setenv(k, v)
    if name.startswith("tail"):
        monkeypatch.setenv("GETT_FORCE_TILE", TAIL_TILE[dtype])
    w = wl.Workload(800 + case, name, "f32" if dtype == np.float32 else "f64", *modes, ext,
                    alpha=-0.75, beta=1.25)
    host, tA, tB, C0 = device_inputs(gpu, w)
    h, d = plan(modes, ext, dtype)
    try:
        assert d["partials"] == "workspace"
        outs = []
        for _ in range(4):
            C = C0.clone()
            run(h, w, tA, tB, C)
            torch.cuda.synchronize()
            outs.append(C)
        for k in range(1, 4):
            assert torch.equal(outs[0], outs[k]), f"call {k} differs from call 0"
        assert compare_whole(outs[0], w, *host) <= TOL[dtype]
    finally:
        g.gett_destroy(h)


def test_workspace_shared_by_plans_of_different_sizes(gpu, monkeypatch):
    """One stream: a small tail plan, then a K-slice plan with more counters
    and slots, then the small plan again -- each result against the oracle
    (the counters are zero again after every call)."""
    import torch
    small = wl.Workload(850, "small_tail", "f64", "a,b", "a,k", "k,b",
                        {"a": 300, "b": 290, "k": 333}, alpha=1.5, beta=-0.5)
    big = wl.Workload(851, "big_slices", "f64", "a,b", "a,k", "k,b",
                      {"a": 700, "b": 650, "k": 3000}, alpha=-1.0, beta=0.5)
    monkeypatch.setenv("GETT_FORCE_TILE", TAIL_TILE[np.float64])
    monkeypatch.setenv("GETT_FORCE_KIND", "3")
    monkeypatch.setenv("GETT_TAIL_WGS", "5")
    hs, ds = plan(("a,b", "a,k", "k,b"), small.extents, np.float64)
    monkeypatch.delenv("GETT_FORCE_KIND")
    monkeypatch.delenv("GETT_TAIL_WGS")
    monkeypatch.setenv("GETT_FORCE_KSLICES", "16")
    hb, db = plan(("a,b", "a,k", "k,b"), big.extents, np.float64)
    try:
        assert ds["kernel"] == "tail" and db["kslices"] == 16
        assert db["workspace_counters"] > ds["workspace_counters"]
        assert db["workspace_bytes"] > ds["workspace_bytes"]
        for w, h in ((small, hs), (big, hb), (small, hs)):
            host, tA, tB, C = device_inputs(gpu, w)
            run(h, w, tA, tB, C)
            torch.cuda.synchronize()
            assert compare_whole(C, w, *host) <= TOL[np.float64], w.name
    finally:
        g.gett_destroy(hs)
        g.gett_destroy(hb)


def test_two_streams_at_once(gpu, monkeypatch):
    """The same K-slice plan launched on two streams back to back: each stream
    has its own workspace, both results match the oracle."""
    import torch
    monkeypatch.setenv("GETT_FORCE_KSLICES", "8")
    w = wl.Workload(860, "two_streams", "f32", "a,b", "a,k", "k,b",
                    {"a": 500, "b": 480, "k": 4000}, alpha=1.0, beta=0.0)
    host, tA, tB, _ = device_inputs(gpu, w)
    h, d = plan(("a,b", "a,k", "k,b"), w.extents, np.float32)
    try:
        assert d["kslices"] == 8 and d["partials"] == "workspace"
        s1, s2 = torch.cuda.Stream(), torch.cuda.Stream()
        C1 = torch.full((w.numel("C"),), float("nan"), device=gpu)
        C2 = torch.full((w.numel("C"),), float("nan"), device=gpu)
        torch.cuda.synchronize()
        for _ in range(3):
            run(h, w, tA, tB, C1, s1)
            run(h, w, tA, tB, C2, s2)
        torch.cuda.synchronize()
        assert torch.equal(C1, C2)
        assert compare_whole(C1, w, *host) <= TOL[np.float32]
    finally:
        g.gett_destroy(h)


def test_c_in_host_memory(gpu, monkeypatch):
    """C in pinned host memory with K slices: the partial tiles live in the
    library's device workspace and C is written with plain stores."""
    import torch
    monkeypatch.setenv("GETT_FORCE_KSLICES", "4")
    w = wl.Workload(870, "host_c", "f64", "a,b", "a,k", "k,b", {"a": 90, "b": 70, "k": 800},
                    alpha=2.0, beta=-1.0)
    host, tA, tB, _ = device_inputs(gpu, w)
    h, d = plan(("a,b", "a,k", "k,b"), w.extents, np.float64)
    try:
        assert d["partials"] == "workspace"
        C = torch.from_numpy(np.asfortranarray(host[2]).reshape(-1, order="F")).pin_memory()
        assert C.is_pinned()
        run(h, w, tA, tB, C)
        torch.cuda.synchronize()
        assert compare_whole(C, w, *host) <= TOL[np.float64]
    finally:
        g.gett_destroy(h)
