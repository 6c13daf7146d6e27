"""GPU parity of method selection (Sec. 6): every candidate method forced in
turn, and the method gett_select_tune keeps, against the oracle on the same
inputs (every beta path, permuted and gapped layouts); the tuned method is
the fastest of those it timed, and TTGT is not timed without its
workspace."""
import json

import numpy as np
import pytest

import oracle
import paper_1607_00145_amd as g
from gpu_util import TOL, make_operand, reference, result_view, split, touched_mask

pytestmark = pytest.mark.gpu
DTYPES = [np.float32, np.float64]
CASES = {
    "ab-ac-cb": (("ab", "ac", "cb"), {"a": 70, "b": 61, "c": 45}),
    "abc-ack-bk": (("abc", "ack", "bk"), {"a": 33, "b": 20, "c": 7, "k": 45}),
    "abij-iejf-faeb": (("a,b,i,j", "i,e,j,f", "f,a,e,b"), {x: 9 for x in "abijef"}),
    "abcijk-dabi-cdjk": (("a,b,c,i,j,k", "d,a,b,i", "c,d,j,k"), {x: 6 for x in "abcdijk"}),
    "abc-bda-dc": (("abc", "bda", "dc"), {"a": 19, "b": 17, "c": 13, "d": 11}),
}


def select_plan(modes, ops, cap=-1):
    C, A, B = ops
    dt = g.GETT_FLOAT32 if C.flat.dtype == np.float32 else g.GETT_FLOAT64
    st, h = g.gett_select_plan(dt, modes[0], C.shape, C.strides, modes[1], A.shape, A.strides,
                               modes[2], B.shape, B.strides, 0, cap)
    assert st == 0, g.gett_status_string(st)
    return h


def run(dev, h, ops, alpha, beta, tune=0, with_workspace=True):
    """Contract (after gett_select_tune over `tune` GETT candidates when
    tune > 0) through the selection plan; returns the whole C buffer."""
    import torch
    C, A, B = ops
    _, nws = g.gett_select_workspace_size(h)
    ws = torch.empty(max(nws, 1), dtype=torch.uint8, device=dev)
    wsp, wsn = (ws.data_ptr(), nws) if with_workspace else (0, 0)
    bufC, _ = C.device(dev)
    bufA, _ = A.device(dev)
    bufB, _ = B.device(dev)
    it = C.flat.itemsize
    pa, pb, pc = (bufA.data_ptr() + A.offset * it, bufB.data_ptr() + B.offset * it,
                  bufC.data_ptr() + C.offset * it)
    stream = torch.cuda.current_stream().cuda_stream
    if tune:
        scratch, _ = C.device(dev)   # tuning overwrites C: time on a copy
        st = g.gett_select_tune(h, tune, pa, pb, scratch.data_ptr() + C.offset * it, wsp, wsn,
                                stream)
        assert st == 0, g.gett_status_string(st)
    st = g.gett_select_contract(h, alpha, pa, pb, beta, pc, wsp, wsn, stream)
    assert st == 0, g.gett_status_string(st)
    torch.cuda.synchronize()
    return bufC.cpu().numpy()


def operands(rng, modes, ext, dtype, kinds, beta):
    shp = lambda m: [ext[x] for x in split(m)]
    C = make_operand(rng, shp(modes[0]), dtype, kinds[0])
    A = make_operand(rng, shp(modes[1]), dtype, kinds[1])
    B = make_operand(rng, shp(modes[2]), dtype, kinds[2])
    inside = touched_mask(C)
    if beta == 0:
        C.flat[inside] = np.nan
    C.flat[~inside] = 7777.0
    return (C, A, B), inside


def check(got_flat, ops, inside, before, ref, dtype):
    assert np.array_equal(got_flat[~inside], before[~inside]), "wrote outside C"
    err = oracle.rel_error(result_view(got_flat, ops[0]), ref)
    assert err <= TOL[dtype], f"rel err {err:.3e}"


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("name", list(CASES))
def test_every_method_forced(gpu, name, dtype):
    modes, ext = CASES[name]
    rng = np.random.default_rng(len(name) * 7 + (dtype == np.float64))
    for alpha, beta, kinds in [(1.0, 0.0, ("dense",) * 3), (-0.5, 1.0, ("permuted", "gapped", "dense")),
                               (1.5, -0.75, ("gapped", "dense", "permuted"))]:
        ops, inside = operands(rng, modes, ext, dtype, kinds, beta)
        before = ops[0].flat.copy()
        ref = reference(modes, ops, alpha, beta)
        h = select_plan(modes, ops)
        try:
            avail = json.loads(g.gett_select_describe(h))["available"]
            for m, key in ((g.GETT_METHOD_GETT, "gett"), (g.GETT_METHOD_TTGT, "ttgt"),
                           (g.GETT_METHOD_LOG, "log")):
                if not avail[key]:
                    continue
                assert g.gett_select_force(h, m) == 0
                ops[0].flat[:] = before
                check(run(gpu, h, ops, alpha, beta), ops, inside, before, ref, dtype)
        finally:
            g.gett_select_destroy(h)


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("name", list(CASES))
def test_tuned_method(gpu, name, dtype):
    modes, ext = CASES[name]
    rng = np.random.default_rng(500 + len(name))
    ops, inside = operands(rng, modes, ext, dtype, ("dense",) * 3, 0.5)
    before = ops[0].flat.copy()
    ref = reference(modes, ops, 1.25, 0.5)
    h = select_plan(modes, ops)
    try:
        check(run(gpu, h, ops, 1.25, 0.5, tune=4), ops, inside, before, ref, dtype)
        d = json.loads(g.gett_select_describe(h))
        assert d["timed"]
        timed = {k: v for k, v in d["ms"].items() if v is not None}
        assert set(timed) == {k for k, v in d["available"].items() if v}
        assert d["method"] == min(timed, key=timed.get)
    finally:
        g.gett_select_destroy(h)


@pytest.mark.parametrize("dtype", DTYPES)
def test_tune_without_workspace_skips_ttgt(gpu, dtype):
    modes, ext = CASES["abcijk-dabi-cdjk"]
    rng = np.random.default_rng(77)
    ops, inside = operands(rng, modes, ext, dtype, ("dense",) * 3, 0.0)
    before = ops[0].flat.copy()
    ref = reference(modes, ops, 1.0, 0.0)
    h = select_plan(modes, ops)
    try:
        assert g.gett_select_workspace_size(h)[1] > 0
        got = run(gpu, h, ops, 1.0, 0.0, tune=2, with_workspace=False)
        d = json.loads(g.gett_select_describe(h))
        assert d["ms"]["ttgt"] is None and d["method"] != "ttgt"
        check(got, ops, inside, before, ref, dtype)
    finally:
        g.gett_select_destroy(h)


@pytest.mark.parametrize("number", [12, 28])
def test_tuned_full_size_sampled(gpu, number):
    """Appendix A contractions 12 (ab-ac-cb) and 28 (abcd-eafb-fdec) in fp32
    at the extents of Table III: the tuned method's C, 1024 sampled elements
    against the oracle."""
    import torch

    import workloads as wl
    from workloads.appendix_a import appendix_workloads
    w = appendix_workloads("f32")[number - 1]
    A, B, _ = wl.make_inputs(w)
    flat = lambda t: torch.from_numpy(np.asfortranarray(t).reshape(-1, order="F")).to(gpu)
    tA, tB = flat(A), flat(B)
    nC = w.numel("C")
    tC = torch.full((nC,), float("nan"), dtype=tA.dtype, device=gpu)
    st, h = g.gett_select_plan(g.GETT_FLOAT32, w.modes_C, w.shape("C"), None, w.modes_A,
                               w.shape("A"), None, w.modes_B, w.shape("B"), None, 0, -1)
    assert st == 0
    try:
        _, nws = g.gett_select_workspace_size(h)
        ws = torch.empty(max(nws, 1), dtype=torch.uint8, device=gpu)
        stream = torch.cuda.current_stream().cuda_stream
        assert g.gett_select_tune(h, 0, tA.data_ptr(), tB.data_ptr(), tC.data_ptr(),
                                  ws.data_ptr(), nws, stream) == 0
        tC.fill_(float("nan"))
        assert g.gett_select_contract(h, 1.0, tA.data_ptr(), tB.data_ptr(), 0.0, tC.data_ptr(),
                                      ws.data_ptr(), nws, stream) == 0
        torch.cuda.synchronize()
        print(w.name, g.gett_select_describe(h))
    finally:
        g.gett_select_destroy(h)
    assert bool(torch.isfinite(tC).all())
    rng = np.random.default_rng(w.seed + 2)
    pts = np.concatenate([rng.integers(0, nC, 1020), [0, 1, nC - 2, nC - 1]])
    got = tC[torch.from_numpy(pts).to(gpu)].cpu().numpy()
    ref = oracle.contract(w.modes_C, w.modes_A, w.modes_B, A, B, 1.0, 0.0, None,
                          shape_C=w.shape("C"), points=pts)
    assert oracle.rel_error(got, ref) <= TOL[np.float32]
