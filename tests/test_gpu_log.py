"""GPU parity of Loops-over-GEMM (Sec. 5) against the oracle, with the
contraction bar of the GETT tests.  Contractions LoG cannot handle
(Listing 7) are checked to be refused."""
import json

import numpy as np
import pytest

import oracle
import paper_1607_00145_amd as g
import workloads as wl
from gpu_util import TOL, make_operand, reference, result_view, split, touched_mask

pytestmark = pytest.mark.gpu
DTYPES = [np.float32, np.float64]


def run_log(dev, modes, ops, alpha, beta):
    import torch
    mc, ma, mb = modes
    C, A, B = ops
    dt = g.GETT_FLOAT32 if C.flat.dtype == np.float32 else g.GETT_FLOAT64
    st, h = g.gett_log_plan(dt, mc, C.shape, C.strides, ma, A.shape, A.strides, mb, B.shape,
                            B.strides)
    if st == g.GETT_ERROR_NOT_SUPPORTED:
        return None, None
    assert st == 0, g.gett_status_string(st)
    try:
        bufC, _ = C.device(dev)
        bufA, _ = A.device(dev)
        bufB, _ = B.device(dev)
        it = C.flat.itemsize
        st = g.gett_log_contract(h, alpha, bufA.data_ptr() + A.offset * it,
                                 bufB.data_ptr() + B.offset * it, beta,
                                 bufC.data_ptr() + C.offset * it,
                                 torch.cuda.current_stream().cuda_stream)
        assert st == 0, g.gett_status_string(st)
        torch.cuda.synchronize()
        return bufC.cpu().numpy(), json.loads(g.gett_log_describe(h))
    finally:
        g.gett_log_destroy(h)


def check_log(dev, rng, modes, shapes, dtype, alpha, beta, kinds=("dense",) * 3):
    C = make_operand(rng, shapes[0], dtype, kinds[0])
    A = make_operand(rng, shapes[1], dtype, kinds[1])
    B = make_operand(rng, shapes[2], dtype, kinds[2])
    inside = touched_mask(C)
    if beta == 0:
        C.flat[inside] = np.nan
    C.flat[~inside] = 7777.0
    before = C.flat.copy()
    got_flat, d = run_log(dev, modes, (C, A, B), alpha, beta)
    if got_flat is None:
        return None
    ref = reference(modes, (C, A, B), alpha, beta)
    assert np.array_equal(got_flat[~inside], before[~inside]), "wrote outside C"
    err = oracle.rel_error(result_view(got_flat, C), ref)
    assert err <= TOL[dtype], f"rel err {err:.3e} for {modes} {shapes} {d}"
    return d


@pytest.mark.parametrize("seed", range(24))
@pytest.mark.parametrize("dtype", DTYPES)
def test_log_random(gpu, seed, dtype):
    rng = np.random.default_rng(65_000 + seed)
    mc, ma, mb, ext = wl.random_problem(rng, max_rank=6, max_ext=7,
                                        allow_empty_sets=(seed % 6 == 5))
    shp = lambda m: [ext[x] for x in split(m)]
    kinds = tuple(rng.choice(["dense", "gapped", "permuted"]) for _ in range(3))
    alpha = float(rng.choice([1.0, -0.75, 2.5]))
    beta = float(rng.choice([0.0, 1.0, -1.25]))
    check_log(gpu, rng, (mc, ma, mb), (shp(mc), shp(ma), shp(mb)), dtype, alpha, beta, kinds)


@pytest.mark.parametrize("dtype", DTYPES)
def test_log_listing8_structure(gpu, dtype):
    """The contraction of Listing 8 at extent 9: batched over k, looped over c."""
    rng = np.random.default_rng(66_000)
    shp = lambda m: [9] * len(m)
    d = check_log(gpu, rng, ("abcijk", "ijmc", "mkab"), (shp("abcijk"), shp("ijmc"), shp("mkab")),
                  dtype, 1.0, 0.5)
    assert d is not None and d["gemm_calls"] == 9


@pytest.mark.parametrize("dtype", DTYPES)
def test_log_contracted_loops_accumulate(gpu, dtype):
    """Two contracted indices: one is the GEMM's k, the other a host loop whose
    GEMMs add into the same slice (beta once)."""
    rng = np.random.default_rng(66_100)
    ext = {"a": 17, "b": 13, "k": 6, "l": 5}
    shp = lambda m: [ext[x] for x in m]
    # k, l adjacent in A but reversed in B: no super-index; B's stride-one l is the GEMM's k
    d = check_log(gpu, rng, ("ab", "akl", "lkb"), (shp("ab"), shp("akl"), shp("lkb")), dtype,
                  1.5, -0.5, ("dense", "gapped", "dense"))
    assert d is not None and d["contracted_loops"] == ["k"] and d["gemm"]["k_index"] == "l"


SCALED = {1: {"a": 20, "b": 9, "c": 13, "k": 17},
          2: {"a": 20, "b": 21, "c": 9, "d": 19, "e": 16},
          3: {"a": 7, "b": 9, "i": 10, "j": 6, "e": 11, "f": 5},
          4: {"a": 5, "b": 6, "c": 7, "d": 24, "i": 4, "j": 3, "k": 5},
          5: {"m1": 9, "m2": 10, "n1": 11, "n2": 7, "k1": 12, "k2": 6}}


@pytest.mark.parametrize("number", [1, 2, 3, 4, 5])
def test_log_workloads_scaled(gpu, number):
    w = wl.scaled(wl.WORKLOADS[number - 1], SCALED[number])
    rng = np.random.default_rng(w.seed + 6)
    d = check_log(gpu, rng, (w.modes_C, w.modes_A, w.modes_B),
                  (w.shape("C"), w.shape("A"), w.shape("B")), w.np_dtype, w.alpha, w.beta)
    assert d is not None


@pytest.mark.parametrize("variant", ["a", "b"])
@pytest.mark.parametrize("k", [8, 1024])
def test_log_fig11_sampled(gpu, variant, k):
    import torch
    w = wl.fig11(variant, k, "f32")
    A, B, _ = wl.make_inputs(w)
    flat = lambda t: torch.from_numpy(np.asfortranarray(t).reshape(-1, order="F")).to(gpu)
    tA, tB = flat(A), flat(B)
    nC = w.numel("C")
    tC = torch.full((nC,), float("nan"), dtype=tA.dtype, device=gpu)
    st, h = g.gett_log_plan(g.GETT_FLOAT32, w.modes_C, w.shape("C"), None, w.modes_A,
                            w.shape("A"), None, w.modes_B, w.shape("B"), None)
    assert st == 0
    try:
        st = g.gett_log_contract(h, 1.0, tA.data_ptr(), tB.data_ptr(), 0.0, tC.data_ptr(),
                                 torch.cuda.current_stream().cuda_stream)
        assert st == 0
        torch.cuda.synchronize()
    finally:
        g.gett_log_destroy(h)
    assert bool(torch.isfinite(tC).all())
    rng = np.random.default_rng(w.seed + 3)
    pts = np.concatenate([rng.integers(0, nC, 2045), [0, nC // 2, nC - 1]])
    got = tC[torch.from_numpy(pts).to(gpu)].cpu().numpy()
    ref = oracle.contract(w.modes_C, w.modes_A, w.modes_B, A, B, 1.0, 0.0, None,
                          shape_C=w.shape("C"), points=pts)
    assert oracle.rel_error(got, ref) <= TOL[np.float32]


@pytest.mark.parametrize("dtype", DTYPES)
def test_log_alpha_zero_and_empty_sum(gpu, dtype):
    rng = np.random.default_rng(67_000)
    ext = {"a": 9, "b": 8, "c": 7, "k": 6}
    shp = lambda m: [ext[x] for x in m]
    check_log(gpu, rng, ("abc", "akc", "kb"), (shp("abc"), shp("akc"), shp("kb")), dtype, 0.0,
              -2.0, ("gapped",) * 3)
    ext["k"] = 0
    check_log(gpu, rng, ("abc", "akc", "kb"), (shp("abc"), shp("akc"), shp("kb")), dtype, 1.0,
              0.5, ("gapped",) * 3)
