"""GPU parity of K slices: several workgroups share one tile's contracted
range; their partial tiles are summed in slice order through the library's
workspace.  Against the oracle for forced slice counts on random
contractions with long contracted sets, integer inputs (exact whatever the
order of the additions), every beta path (beta = 0 with NaN in C, beta = 1
with no scaling pass, any other beta), alpha = 0, more slices than K boxes,
and the model's own choice on a small output with a deep contracted set."""
import json

import numpy as np
import pytest

import paper_1607_00145_amd as g
import workloads as wl
from gpu_util import split
from test_gpu_parity import check_case

pytestmark = pytest.mark.gpu
DTYPES = [np.float32, np.float64]


def shapes(modes, ext):
    return tuple([ext[x] for x in split(m)] for m in modes)


def describe(modes, ext, dtype, flags=0):
    code = g.GETT_FLOAT32 if dtype == np.float32 else g.GETT_FLOAT64
    sh = shapes(modes, ext)
    st, h = g.gett_plan(code, modes[0], sh[0], None, modes[1], sh[1], None, modes[2], sh[2],
                        None, flags)
    assert st == 0
    try:
        return json.loads(g.gett_plan_describe(h))
    finally:
        g.gett_destroy(h)


# small C, long contracted sets (the shape of Appendix A's ab-acd-dbc and
# abc-adec-ebd, reduced), with ragged tails everywhere
DEEP = {
    "ab-acd-dbc": (("a,b", "a,c,d", "d,b,c"), {"a": 45, "b": 38, "c": 29, "d": 37}),
    "abc-adec-ebd": (("a,b,c", "a,d,e,c", "e,b,d"), {"a": 21, "b": 13, "c": 6, "d": 17, "e": 19}),
    "ab-ak-kb": (("a,b", "a,k", "k,b"), {"a": 33, "b": 70, "k": 1000}),
}


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("slices", [2, 3, 8, 64])
@pytest.mark.parametrize("name", list(DEEP))
def test_forced_slices(gpu, monkeypatch, name, slices, dtype):
    monkeypatch.setenv("GETT_FORCE_KSLICES", str(slices))
    modes, ext = DEEP[name]
    d = describe(modes, ext, dtype)
    assert d["kslices"] == slices
    assert d["partials"] == "workspace"
    rng = np.random.default_rng(1000 * slices + len(name))
    for alpha, beta in [(1.0, 0.0), (-0.75, 1.0), (1.5, -0.5)]:
        check_case(gpu, rng, modes, shapes(modes, ext), dtype, alpha, beta)


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("name", list(DEEP))
def test_slices_integer_inputs_exact(gpu, monkeypatch, name, dtype):
    monkeypatch.setenv("GETT_FORCE_KSLICES", "16")
    modes, ext = DEEP[name]
    rng = np.random.default_rng(3)
    for beta in (0.0, 1.0, 2.0):
        got, ref = check_case(gpu, rng, modes, shapes(modes, ext), dtype, 1.0, beta, dist="int")
        np.testing.assert_array_equal(got.astype(np.float64), ref.out64)


@pytest.mark.parametrize("dtype", DTYPES)
def test_slices_with_gapped_and_permuted_layouts(gpu, monkeypatch, dtype):
    monkeypatch.setenv("GETT_FORCE_KSLICES", "5")
    modes, ext = DEEP["ab-acd-dbc"]
    rng = np.random.default_rng(17)
    for kinds in [("gapped",) * 3, ("permuted", "gapped", "dense"), ("dense", "permuted", "permuted")]:
        check_case(gpu, rng, modes, shapes(modes, ext), dtype, 0.5, 0.25, kinds=kinds)


@pytest.mark.parametrize("dtype", DTYPES)
def test_more_slices_than_boxes(gpu, monkeypatch, dtype):
    """Slices beyond the number of K boxes get no boxes and add zero."""
    monkeypatch.setenv("GETT_FORCE_KSLICES", "256")
    modes, ext = (("a,b", "a,k", "k,b"), {"a": 40, "b": 50, "k": 100})
    d = describe(modes, ext, dtype)
    assert d["kslices"] == 256 and d["kbox"]["steps"] < 256
    rng = np.random.default_rng(5)
    check_case(gpu, rng, modes, shapes(modes, ext), dtype, 1.0, -1.0)
    check_case(gpu, rng, modes, shapes(modes, ext), dtype, 2.0, 0.0)


@pytest.mark.parametrize("dtype", DTYPES)
def test_slices_alpha_zero(gpu, monkeypatch, dtype):
    """alpha = 0 on a sliced plan: C <- beta * C, A and B not read."""
    monkeypatch.setenv("GETT_FORCE_KSLICES", "8")
    modes, ext = DEEP["ab-ak-kb"]
    rng = np.random.default_rng(9)
    for beta in (0.0, 1.5):
        check_case(gpu, rng, modes, shapes(modes, ext), dtype, 0.0, beta)


@pytest.mark.parametrize("dtype", DTYPES)
def test_model_slices_small_output_deep_k(gpu, dtype):
    """The model takes K slices for a small C over a long contracted set, and
    not with the deterministic flag; both agree with the oracle."""
    modes, ext = (("a,b", "a,c,d", "d,b,c"), {"a": 96, "b": 94, "c": 94, "d": 96})
    assert describe(modes, ext, dtype)["kslices"] > 1
    assert describe(modes, ext, dtype, g.GETT_FLAG_DETERMINISTIC)["kslices"] == 1
    rng = np.random.default_rng(21)
    check_case(gpu, rng, modes, shapes(modes, ext), dtype, 1.25, 0.5)
    check_case(gpu, rng, modes, shapes(modes, ext), dtype, 1.0, 0.0,
               flags=g.GETT_FLAG_DETERMINISTIC)


@pytest.mark.parametrize("number", [1, 2, 3, 4, 5])
def test_workload_structures_sliced(gpu, monkeypatch, number):
    """Every workload's index structure (reduced, ragged) with K slices forced."""
    from test_gpu_parity import SCALED
    monkeypatch.setenv("GETT_FORCE_KSLICES", "4")
    w = wl.scaled(wl.WORKLOADS[number - 1], SCALED[number])
    dtype = np.float32 if w.dtype == "f32" else np.float64
    rng = np.random.default_rng(number)
    check_case(gpu, rng, (w.modes_C, w.modes_A, w.modes_B),
               (w.shape("C"), w.shape("A"), w.shape("B")), dtype, w.alpha, w.beta)


@pytest.mark.parametrize("dtype", ["f32", "f64"])
@pytest.mark.parametrize("number", [13, 14, 19])
def test_appendix_sliced_full_size(gpu, number, dtype):
    """The model's sliced plans at the paper's extents (Appendix A
    contractions 13, 14, 19; Tables III / IV), alpha 1.5 and beta -0.5 on a
    filled C (the beta pass runs), 1024 sampled elements against the oracle."""
    import torch

    import oracle
    from gpu_util import TOL
    from workloads.appendix_a import appendix_workloads
    w = appendix_workloads(dtype)[number - 1]
    npdt = np.float32 if dtype == "f32" else np.float64
    A, B, _ = wl.make_inputs(w)
    rng = np.random.default_rng(w.seed + 7)
    C0 = rng.uniform(-1, 1, w.numel("C")).astype(npdt)
    flat = lambda t: torch.from_numpy(np.asfortranarray(t).reshape(-1, order="F")).to(gpu)
    tA, tB, tC = flat(A), flat(B), torch.from_numpy(C0.copy()).to(gpu)
    code = g.GETT_FLOAT32 if dtype == "f32" else g.GETT_FLOAT64
    st, h = g.gett_plan(code, w.modes_C, w.shape("C"), None, w.modes_A, w.shape("A"), None,
                        w.modes_B, w.shape("B"), None, 0)
    assert st == 0
    try:
        assert json.loads(g.gett_plan_describe(h))["kslices"] > 1
        st = g.gett_contract(h, 1.5, tA.data_ptr(), tB.data_ptr(), -0.5, tC.data_ptr(),
                             torch.cuda.current_stream().cuda_stream)
        assert st == 0
        torch.cuda.synchronize()
    finally:
        g.gett_destroy(h)
    nC = w.numel("C")
    pts = np.concatenate([rng.integers(0, nC, 1020), [0, 1, nC - 2, nC - 1]])
    got = tC[torch.from_numpy(pts).to(gpu)].cpu().numpy()
    Cin = C0.reshape(w.shape("C"), order="F")
    ref = oracle.contract(w.modes_C, w.modes_A, w.modes_B, A, B, 1.5, -0.5, Cin,
                          shape_C=w.shape("C"), points=pts)
    assert oracle.rel_error(got, ref) <= TOL[npdt]
