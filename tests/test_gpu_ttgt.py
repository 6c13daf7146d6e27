"""GPU parity of the Eq. 4 transposition kernel and of TTGT (Sec. 4) against
the oracle.

Transposition bar: alpha 1, beta 0 must be bit-exact (a pure copy); otherwise
|got - ref| <= 2 u (|alpha a| + |beta b|) with u the unit roundoff of the
type (one rounding of alpha * a, one of the sum).  Elements of the output
buffer outside the output tensor must be untouched.  TTGT uses the
contraction bar of the GETT tests (it computes the same contraction)."""
import json

import numpy as np
import pytest

import oracle
import paper_1607_00145_amd as g
import workloads as wl
from gpu_util import TOL, make_operand, reference, result_view, split, touched_mask

pytestmark = pytest.mark.gpu
DTYPES = [np.float32, np.float64]
TOL_T = {np.float32: 2 * 2.0 ** -24, np.float64: 2 * 2.0 ** -53}


def run_transpose(dev, In, Out, perm, alpha, beta, dtype):
    import torch
    it = In.flat.itemsize
    bufI, _ = In.device(dev)
    bufO, _ = Out.device(dev)
    sout = [0] * len(perm)
    for j, d in enumerate(perm):
        sout[d] = Out.strides[j]
    dt = g.GETT_FLOAT32 if dtype == np.float32 else g.GETT_FLOAT64
    st = g.gett_transpose(dt, In.shape, In.strides, sout, alpha, bufI.data_ptr() + In.offset * it,
                          beta, bufO.data_ptr() + Out.offset * it,
                          torch.cuda.current_stream().cuda_stream)
    assert st == 0, g.gett_status_string(st)
    torch.cuda.synchronize()
    return bufO.cpu().numpy()


def check_transpose(dev, rng, shape, perm, dtype, alpha, beta, kinds=("dense", "dense")):
    In = make_operand(rng, shape, dtype, kinds[0])
    Out = make_operand(rng, [shape[p] for p in perm], dtype, kinds[1])
    inside = touched_mask(Out)
    if beta == 0:
        Out.flat[inside] = np.nan
    Out.flat[~inside] = 4321.0
    before = Out.flat.copy()
    ref = oracle.transpose(In.view, perm, alpha, beta, Out.view if beta != 0 else None)
    got_flat = run_transpose(dev, In, Out, perm, alpha, beta, dtype)
    assert np.array_equal(got_flat[~inside], before[~inside]), "wrote outside the output"
    got = result_view(got_flat, Out).astype(np.float64)
    if alpha == 1.0 and beta == 0.0:
        assert np.array_equal(got, ref.out64), (shape, perm)
    else:
        err = np.abs(got - ref.out64)
        assert np.all(err <= TOL_T[dtype] * ref.den64), (shape, perm, float(err.max()))


@pytest.mark.parametrize("seed", range(20))
@pytest.mark.parametrize("dtype", DTYPES)
def test_transpose_random(gpu, seed, dtype):
    rng = np.random.default_rng(60_000 + seed)
    rank = int(rng.integers(0, 7))
    shape = [int(rng.integers(1, 9)) for _ in range(rank)]
    perm = list(rng.permutation(rank))
    kinds = tuple(rng.choice(["dense", "gapped", "permuted"]) for _ in range(2))
    alpha = float(rng.choice([1.0, -0.5, 2.0, 0.0]))
    beta = float(rng.choice([0.0, 1.0, -1.5]))
    check_transpose(gpu, rng, shape, perm, dtype, alpha, beta, kinds)


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("shape,perm", [
    ([130, 70], [1, 0]),              # several tiles, ragged in both directions
    ([64, 64], [1, 0]),               # exactly one tile
    ([200, 3, 50], [2, 1, 0]),
    ([5, 7, 9, 11], [3, 0, 2, 1]),    # compound tile sides
    ([3, 300, 2], [1, 2, 0]),
    ([1000], [0]),                    # one index: an axpby
    ([70, 90], [0, 1]),               # the output's stride-one index is the input's
    ([2, 2, 2, 2, 2, 2, 2, 2, 2, 2, 2, 2], [11, 10, 9, 8, 7, 6, 5, 4, 3, 2, 1, 0]),
    ([132, 68], [1, 0]),              # 16-byte reads and writes, ragged tiles
    ([68, 5, 7], [0, 2, 1]),          # vector writes along the shared stride-one index
    ([8, 12, 20], [2, 0, 1]),         # vector reads over a compound tile side
    ([36, 6, 10], [1, 2, 0]),
    ([40, 36, 12, 8], [1, 0, 3, 2]),  # batched pair swaps: the output's stride-one
    ([20, 140, 6], [1, 0, 2]),        # index is second by input stride (not in P)
    ([8, 3, 44, 12], [2, 1, 0, 3]),
    ([35001, 300], [1, 0]),           # more P tiles than half the resident workgroups:
    ([33001, 130, 2], [1, 0, 2]),     # bands of P tiles, the last one short
])
def test_transpose_shapes(gpu, dtype, shape, perm):
    rng = np.random.default_rng(61_000 + sum(shape))
    check_transpose(gpu, rng, shape, perm, dtype, 1.0, 0.0)
    check_transpose(gpu, rng, shape, perm, dtype, -0.75, 1.25, ("gapped", "gapped"))


# ------------------------------------------------------------------ TTGT ---

def run_ttgt(dev, modes, ops, alpha, beta, cap=-1):
    import torch
    mc, ma, mb = modes
    C, A, B = ops
    dt = g.GETT_FLOAT32 if C.flat.dtype == np.float32 else g.GETT_FLOAT64
    st, h = g.gett_ttgt_plan(dt, mc, C.shape, C.strides, ma, A.shape, A.strides, mb, B.shape,
                             B.strides, cap)
    assert st == 0, g.gett_status_string(st)
    try:
        _, nws = g.gett_ttgt_workspace_size(h)
        ws = torch.empty(max(nws, 1), dtype=torch.uint8, device=dev)
        bufC, _ = C.device(dev)
        bufA, _ = A.device(dev)
        bufB, _ = B.device(dev)
        it = C.flat.itemsize
        st = g.gett_ttgt_contract(h, alpha, bufA.data_ptr() + A.offset * it,
                                  bufB.data_ptr() + B.offset * it, beta,
                                  bufC.data_ptr() + C.offset * it, ws.data_ptr(), nws,
                                  torch.cuda.current_stream().cuda_stream)
        assert st == 0, g.gett_status_string(st)
        torch.cuda.synchronize()
        return bufC.cpu().numpy(), json.loads(g.gett_ttgt_describe(h))
    finally:
        g.gett_ttgt_destroy(h)


def check_ttgt(dev, rng, modes, shapes, dtype, alpha, beta, kinds=("dense",) * 3):
    C = make_operand(rng, shapes[0], dtype, kinds[0])
    A = make_operand(rng, shapes[1], dtype, kinds[1])
    B = make_operand(rng, shapes[2], dtype, kinds[2])
    inside = touched_mask(C)
    if beta == 0:
        C.flat[inside] = np.nan
    C.flat[~inside] = 7777.0
    before = C.flat.copy()
    ref = reference(modes, (C, A, B), alpha, beta)
    got_flat, d = run_ttgt(dev, modes, (C, A, B), alpha, beta)
    assert np.array_equal(got_flat[~inside], before[~inside]), "wrote outside C"
    err = oracle.rel_error(result_view(got_flat, C), ref)
    assert err <= TOL[dtype], f"rel err {err:.3e} for {modes} {shapes} {d}"
    return d


@pytest.mark.parametrize("seed", range(24))
@pytest.mark.parametrize("dtype", DTYPES)
def test_ttgt_random(gpu, seed, dtype):
    rng = np.random.default_rng(62_000 + seed)
    mc, ma, mb, ext = wl.random_problem(rng, max_rank=6, max_ext=7,
                                        allow_empty_sets=(seed % 6 == 5))
    shp = lambda m: [ext[x] for x in split(m)]
    kinds = tuple(rng.choice(["dense", "gapped", "permuted"]) for _ in range(3))
    alpha = float(rng.choice([1.0, -0.75, 2.5]))
    beta = float(rng.choice([0.0, 1.0, -1.25]))
    check_ttgt(gpu, rng, (mc, ma, mb), (shp(mc), shp(ma), shp(mb)), dtype, alpha, beta, kinds)


@pytest.mark.parametrize("dtype", DTYPES)
def test_ttgt_listing6_and_gemm(gpu, dtype):
    rng = np.random.default_rng(63_000)
    ext = {"a": 33, "b": 20, "c": 7, "k": 45}
    shp = lambda m: [ext[x] for x in m]
    d = check_ttgt(gpu, rng, ("abc", "ack", "bk"), (shp("abc"), shp("ack"), shp("bk")), dtype,
                   1.5, -0.5)
    assert d["transposed"] == ["C"]
    ext = {"m": 130, "n": 70, "k": 90}
    shp = lambda m: [ext[x] for x in m]
    for ma, mb in (("mk", "kn"), ("km", "kn"), ("mk", "nk"), ("km", "nk")):
        d = check_ttgt(gpu, rng, ("mn", ma, mb), (shp("mn"), shp(ma), shp(mb)), dtype, 1.0, 1.0)
        assert d["transposed"] == []


SCALED = {1: {"a": 20, "b": 9, "c": 13, "k": 17},
          2: {"a": 20, "b": 21, "c": 9, "d": 19, "e": 16},
          3: {"a": 7, "b": 9, "i": 10, "j": 6, "e": 11, "f": 5},
          4: {"a": 5, "b": 6, "c": 7, "d": 24, "i": 4, "j": 3, "k": 5},
          5: {"m1": 9, "m2": 10, "n1": 11, "n2": 7, "k1": 12, "k2": 6}}


@pytest.mark.parametrize("number", [1, 2, 3, 4, 5])
def test_ttgt_workloads_scaled(gpu, number):
    w = wl.scaled(wl.WORKLOADS[number - 1], SCALED[number])
    rng = np.random.default_rng(w.seed + 5)
    check_ttgt(gpu, rng, (w.modes_C, w.modes_A, w.modes_B),
               (w.shape("C"), w.shape("A"), w.shape("B")), w.np_dtype, w.alpha, w.beta)


@pytest.mark.parametrize("number", [1, 2, 3, 4, 5])
def test_ttgt_workloads_full_size_sampled(gpu, number):
    """Full-size workloads as the benchmark runs them; 4096 sampled elements."""
    import torch
    w = wl.WORKLOADS[number - 1]
    A, B, Cin = wl.make_inputs(w)
    flat = lambda t: torch.from_numpy(np.asfortranarray(t).reshape(-1, order="F")).to(gpu)
    tA, tB = flat(A), flat(B)
    nC = w.numel("C")
    tC = flat(Cin) if Cin is not None else torch.full((nC,), float("nan"), dtype=tA.dtype,
                                                      device=gpu)
    dt = g.GETT_FLOAT32 if w.dtype == "f32" else g.GETT_FLOAT64
    st, h = g.gett_ttgt_plan(dt, w.modes_C, w.shape("C"), None, w.modes_A, w.shape("A"), None,
                             w.modes_B, w.shape("B"), None, -1)
    assert st == 0
    try:
        _, nws = g.gett_ttgt_workspace_size(h)
        ws = torch.empty(max(nws, 1), dtype=torch.uint8, device=gpu)
        st = g.gett_ttgt_contract(h, w.alpha, tA.data_ptr(), tB.data_ptr(), w.beta, tC.data_ptr(),
                                  ws.data_ptr(), nws, torch.cuda.current_stream().cuda_stream)
        assert st == 0
        torch.cuda.synchronize()
    finally:
        g.gett_ttgt_destroy(h)
    if Cin is None:
        assert bool(torch.isfinite(tC).all())
    rng = np.random.default_rng(w.seed + 98)
    pts = np.concatenate([rng.integers(0, nC, 4091), [0, 1, nC // 2, nC - 2, nC - 1]])
    got = tC[torch.from_numpy(pts).to(gpu)].cpu().numpy()
    ref = oracle.contract(w.modes_C, w.modes_A, w.modes_B, A, B, w.alpha, w.beta, Cin,
                          shape_C=w.shape("C"), points=pts)
    err = oracle.rel_error(got, ref)
    assert err <= TOL[w.np_dtype], f"{w.name}: rel err {err:.3e}"


@pytest.mark.parametrize("dtype", DTYPES)
def test_ttgt_alpha_zero_and_empty_sum(gpu, dtype):
    rng = np.random.default_rng(64_000)
    ext = {"a": 9, "b": 8, "c": 7, "k": 6}
    shp = lambda m: [ext[x] for x in m]
    check_ttgt(gpu, rng, ("abc", "akc", "kb"), (shp("abc"), shp("akc"), shp("kb")), dtype, 0.0,
               -2.0, ("gapped",) * 3)
    ext["k"] = 0
    check_ttgt(gpu, rng, ("abc", "akc", "kb"), (shp("abc"), shp("akc"), shp("kb")), dtype, 1.0,
               0.5, ("gapped",) * 3)


def test_transpose_largest_supported_offsets(gpu):
    """An 8.6 GB fp32 matrix (offsets just below 2^31 - 1) transposed: every
    output element written, sampled elements exact."""
    import torch
    m, n = 65536, 32767
    src = torch.rand(m * n, dtype=torch.float32, device=gpu)
    dst = torch.full((m * n,), float("nan"), dtype=torch.float32, device=gpu)
    st = g.gett_transpose(g.GETT_FLOAT32, [m, n], [1, m], [n, 1], 1.0, src.data_ptr(), 0.0,
                          dst.data_ptr(), torch.cuda.current_stream().cuda_stream)
    assert st == 0
    torch.cuda.synchronize()
    assert bool(torch.isfinite(dst).all())
    rng = np.random.default_rng(71_000)
    i = np.concatenate([rng.integers(0, m, 2000), [0, m - 1, m - 1, 0]])
    j = np.concatenate([rng.integers(0, n, 2000), [0, n - 1, 0, n - 1]])
    a = src[torch.from_numpy(i + j * m).to(gpu)].cpu().numpy()
    b = dst[torch.from_numpy(j + i * n).to(gpu)].cpu().numpy()
    assert np.array_equal(a, b)
    assert g.gett_transpose(g.GETT_FLOAT32, [m, n + 1], [1, m], [n + 1, 1], 1.0, src.data_ptr(),
                            0.0, dst.data_ptr(), 0) == g.GETT_ERROR_NOT_SUPPORTED
