"""GPU tests of the plan-time candidate search (gett_plan_tune): the tuned
plan still matches the oracle, the timings are reported, and the winner is
remembered for later plans of the same descriptor."""
import json

import numpy as np
import pytest

import oracle
import paper_1607_00145_amd as g
import workloads as wl
from gpu_util import TOL, make_operand, reference, result_view, split

pytestmark = pytest.mark.gpu


def kind_of(d):
    """The candidate kind of a described plan."""
    return "kslices" if d["kslices"] > 1 else d["kernel"]


def _plan(modes, ops, dt):
    mc, ma, mb = modes
    C, A, B = ops
    st, h = g.gett_plan(dt, mc, C.shape, C.strides, ma, A.shape, A.strides, mb, B.shape,
                        B.strides, 0)
    assert st == 0, g.gett_status_string(st)
    return h


@pytest.mark.parametrize("name,ext", [("bw4x3_fp32", {"a": 40, "b": 36, "c": 50, "d": 44}),
                                      ("cc4x4_fp64", {m: 14 for m in "abij"}),
                                      ("gemm4_fp32", {m: 24 for m in ["m1", "m2", "n1", "n2"]})])
def test_tuned_plan_matches_oracle(gpu, name, ext):
    import torch
    w = wl.scaled(wl.BY_NAME[name], ext, "_tune")
    dtype = w.np_dtype
    dt = g.GETT_FLOAT32 if w.dtype == "f32" else g.GETT_FLOAT64
    rng = np.random.default_rng(50_000 + w.number)
    modes = (w.modes_C, w.modes_A, w.modes_B)
    C = make_operand(rng, w.shape("C"), dtype, "gapped")
    A = make_operand(rng, w.shape("A"), dtype, "permuted")
    B = make_operand(rng, w.shape("B"), dtype, "dense")
    h = _plan(modes, (C, A, B), dt)
    try:
        before = json.loads(g.gett_plan_describe(h))
        assert before["tile"]["chosen_by"] in ("model", "remembered")
        bufC, _ = C.device(gpu)
        bufA, _ = A.device(gpu)
        bufB, _ = B.device(gpu)
        it = C.flat.itemsize
        stream = torch.cuda.current_stream().cuda_stream
        k = 4
        st = g.gett_plan_tune(h, k, bufA.data_ptr(), bufB.data_ptr(), bufC.data_ptr(), stream)
        assert st == 0, g.gett_status_string(st)
        d = json.loads(g.gett_plan_describe(h))
        assert d["tile"]["chosen_by"] == "tuned"
        timed = d["tuning"]
        assert len(timed) == min(k, len(before["candidates"]))
        assert [(t["tile"], t["kind"]) for t in timed] == \
            [(c["tile"], c["kind"]) for c in before["candidates"][:len(timed)]]
        best = min(timed, key=lambda t: t["measured_us"])
        assert (d["tile"]["id"], kind_of(d)) == (best["tile"], best["kind"])
        assert all(t["measured_us"] > 0 for t in timed)
        # the tuned plan, with the caller's alpha and beta, against the oracle
        Cin = C.flat.copy()
        bufC.copy_(torch.from_numpy(Cin))
        st = g.gett_contract(h, w.alpha, bufA.data_ptr(), bufB.data_ptr(), w.beta,
                             bufC.data_ptr(), stream)
        assert st == 0
        torch.cuda.synchronize()
        got = result_view(bufC.cpu().numpy(), C)
        ref = reference(modes, (C, A, B), w.alpha, w.beta)
        err = oracle.rel_error(got, ref)
        assert err <= TOL[dtype], err
        # a new plan of the same descriptor starts from the tuned choice
        h2 = _plan(modes, (C, A, B), dt)
        d2 = json.loads(g.gett_plan_describe(h2))
        g.gett_destroy(h2)
        assert d2["tile"]["chosen_by"] == "remembered"
        assert (d2["tile"]["id"], kind_of(d2)) == (d["tile"]["id"], kind_of(d))
        assert d2["kslices"] == d["kslices"]
        # another layout of C is another descriptor
        C2 = make_operand(rng, w.shape("C"), dtype, "dense")
        h3 = _plan(modes, (C2, A, B), dt)
        d3 = json.loads(g.gett_plan_describe(h3))
        g.gett_destroy(h3)
        assert d3["tile"]["chosen_by"] == "model"
    finally:
        g.gett_destroy(h)


def test_tune_one_candidate_keeps_the_model_choice(gpu):
    import torch
    rng = np.random.default_rng(50_100)
    modes = ("a,b,c", "a,k,c", "k,b")
    C = make_operand(rng, [33, 20, 7], np.float64)
    A = make_operand(rng, [33, 29, 7], np.float64)
    B = make_operand(rng, [29, 20], np.float64)
    h = _plan(modes, (C, A, B), g.GETT_FLOAT64)
    try:
        d0 = json.loads(g.gett_plan_describe(h))
        bufC, _ = C.device(gpu)
        bufA, _ = A.device(gpu)
        bufB, _ = B.device(gpu)
        st = g.gett_plan_tune(h, 1, bufA.data_ptr(), bufB.data_ptr(), bufC.data_ptr(), 0)
        assert st == 0
        d = json.loads(g.gett_plan_describe(h))
        assert len(d["tuning"]) == 1
        assert (d["tile"]["id"], kind_of(d)) == (d0["tile"]["id"], kind_of(d0))
        # C was overwritten with alpha 1, beta 0
        torch.cuda.synchronize()
        got = result_view(bufC.cpu().numpy(), C)
        ref = reference(modes, (C, A, B), 1.0, 0.0)
        assert oracle.rel_error(got, ref) <= TOL[np.float64]
    finally:
        g.gett_destroy(h)


def test_plan_class_tune(gpu):
    import torch
    a = torch.randn(24, 18, 30, dtype=torch.float32, device=gpu)
    b = torch.randn(30, 26, dtype=torch.float32, device=gpu)
    c = torch.empty(26, 24, 18, dtype=torch.float32, device=gpu)
    p = g.Plan("C[n,i,j] = A[i,j,k] * B[k,n]", C=c, A=a, B=b)
    d = p.tune(a, b, c, max_candidates=3)
    assert d["tile"]["chosen_by"] == "tuned"
    p(a, b, c)
    torch.cuda.synchronize()
    ref = torch.einsum("ijk,kn->nij", a.double().cpu(), b.double().cpu())
    assert torch.allclose(c.double().cpu(), ref, rtol=1e-4, atol=1e-4)
