"""GPU parity: the HIP path (through the C interface) against the oracle.

Bar: max |diff| / (|alpha| * sum_k |a||b| + |beta| * |c|) <= 1e-4 for fp32 and
1e-12 for fp64, element by element; integer-valued inputs must match exactly;
elements of the C buffer that are not part of C must be left untouched."""
import json

import numpy as np
import pytest

import oracle
import paper_1607_00145_amd as g
import workloads as wl
from gpu_util import TOL, Operand, compare_whole, make_operand, reference, result_view, \
    run_gpu, split, touched_mask

pytestmark = pytest.mark.gpu
DTYPES = [np.float32, np.float64]


def check_case(dev, rng, modes, shapes, dtype, alpha, beta, kinds=("dense",) * 3, flags=0,
               dist="uniform", offsets=(0, 0, 0)):
    mc, ma, mb = modes
    C = make_operand(rng, shapes[0], dtype, kinds[0], dist, offsets[0])
    A = make_operand(rng, shapes[1], dtype, kinds[1], dist, offsets[1])
    B = make_operand(rng, shapes[2], dtype, kinds[2], dist, offsets[2])
    inside = touched_mask(C)
    if beta == 0:
        C.flat[inside] = np.nan          # beta == 0 must not read C; every element gets written
    C.flat[~inside] = 7777.0             # canaries in gaps and guard bands
    before = C.flat.copy()
    ref = reference(modes, (C, A, B), alpha, beta)
    got_flat, _ = run_gpu(dev, modes, (C, A, B), alpha, beta, flags)
    assert np.array_equal(got_flat[~inside], before[~inside]), "wrote outside C"
    got = result_view(got_flat, C)
    err = oracle.rel_error(got, ref)
    assert err <= TOL[dtype], f"rel err {err:.3e} for {modes} {shapes}"
    return got, ref


@pytest.mark.parametrize("seed", range(24))
@pytest.mark.parametrize("dtype", DTYPES)
def test_random_contractions(gpu, seed, dtype):
    rng = np.random.default_rng(10_000 + seed)
    mc, ma, mb, ext = wl.random_problem(rng, max_rank=6, max_ext=7,
                                        allow_empty_sets=(seed % 6 == 5))
    shp = lambda m: [ext[x] for x in split(m)]
    kinds = tuple(rng.choice(["dense", "gapped", "permuted"]) for _ in range(3))
    alpha = float(rng.choice([1.0, -0.75, 2.5]))
    beta = float(rng.choice([0.0, 1.0, -1.25]))
    check_case(gpu, rng, (mc, ma, mb), (shp(mc), shp(ma), shp(mb)), dtype, alpha, beta, kinds)


@pytest.mark.parametrize("seed", range(8))
@pytest.mark.parametrize("dtype", DTYPES)
def test_integer_inputs_bit_exact(gpu, seed, dtype):
    """Integer inputs make every partial sum exact: results must be identical."""
    rng = np.random.default_rng(20_000 + seed)
    mc, ma, mb, ext = wl.random_problem(rng, max_rank=6, max_ext=9)
    shp = lambda m: [ext[x] for x in split(m)]
    beta = float(seed % 2)
    got, ref = check_case(gpu, rng, (mc, ma, mb), (shp(mc), shp(ma), shp(mb)), dtype, 1.0, beta,
                          dist="int")
    np.testing.assert_array_equal(got.astype(np.float64), ref.out64)


SCALED = {
    1: {"a": 37, "b": 29, "c": 5, "k": 41},
    2: {"a": 23, "b": 19, "c": 21, "d": 13, "e": 16},
    3: {"a": 11, "b": 13, "i": 12, "j": 14, "e": 9, "f": 17},
    4: {"a": 7, "b": 6, "c": 9, "d": 24, "i": 5, "j": 8, "k": 7},
    5: {"m1": 40, "m2": 6, "n1": 36, "n2": 7, "k1": 10, "k2": 33},
}


@pytest.mark.parametrize("number", [1, 2, 3, 4, 5])
def test_workload_structure_scaled(gpu, number):
    """Each workload's index structure at sizes the oracle checks in full:
    several tiles along each free set and ragged tails everywhere."""
    w = wl.scaled(wl.WORKLOADS[number - 1], SCALED[number])
    rng = np.random.default_rng(w.seed)
    check_case(gpu, rng, (w.modes_C, w.modes_A, w.modes_B),
               (w.shape("C"), w.shape("A"), w.shape("B")), w.np_dtype, w.alpha, w.beta)


@pytest.mark.parametrize("number", [1, 2, 3, 4, 5])
def test_workload_full_size_whole(gpu, number):
    """Full-size workloads in the benchmark's launch configuration, every
    element of C against the oracle (Sec. 7: the naive loop nest as the
    correctness reference).  For beta == 0 C starts as NaN, so an element
    never written would also fail."""
    import torch
    w = wl.WORKLOADS[number - 1]
    A, B, Cin = wl.make_inputs(w)
    dev = gpu
    tA = torch.from_numpy(np.asfortranarray(A).reshape(-1, order="F")).to(dev)
    tB = torch.from_numpy(np.asfortranarray(B).reshape(-1, order="F")).to(dev)
    nC = w.numel("C")
    if Cin is not None:
        tC = torch.from_numpy(np.asfortranarray(Cin).reshape(-1, order="F")).to(dev)
    else:
        tC = torch.full((nC,), float("nan"), dtype=tA.dtype, device=dev)
    dt = g.GETT_FLOAT32 if w.dtype == "f32" else g.GETT_FLOAT64
    st, h = g.gett_plan(dt, w.modes_C, w.shape("C"), None, w.modes_A, w.shape("A"), None,
                        w.modes_B, w.shape("B"), None, 0)
    assert st == 0
    st = g.gett_contract(h, w.alpha, tA.data_ptr(), tB.data_ptr(), w.beta, tC.data_ptr(),
                         torch.cuda.current_stream().cuda_stream)
    assert st == 0
    torch.cuda.synchronize()
    g.gett_destroy(h)
    del tA, tB
    if Cin is None:
        assert bool(torch.isfinite(tC).all()), "some element of C was not written"
    err = compare_whole(tC, w, A, B, Cin)
    print(f"{w.name}: {nC} elements, max rel err {err:.3e}", flush=True)
    assert err <= TOL[w.np_dtype], f"{w.name}: rel err {err:.3e}"


@pytest.mark.parametrize("dtype", DTYPES)
def test_alpha_zero_reads_no_operand(gpu, dtype):
    rng = np.random.default_rng(5)
    modes = ("a,b", "a,k", "k,b")
    C = make_operand(rng, [70, 45], dtype)
    A = make_operand(rng, [70, 33], dtype)
    B = make_operand(rng, [33, 45], dtype)
    A.flat[:] = np.nan
    B.flat[:] = np.nan
    ref = result_view(C.flat, C).astype(np.float64) * -2.0
    got_flat, _ = run_gpu(gpu, modes, (C, A, B), 0.0, -2.0)
    np.testing.assert_array_equal(result_view(got_flat, C).astype(np.float64), ref)


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("flags", [g.GETT_FLAG_SCALAR, g.GETT_FLAG_NO_SWAP,
                                   g.GETT_FLAG_SCALAR | g.GETT_FLAG_NO_SWAP])
def test_flags(gpu, dtype, flags):
    rng = np.random.default_rng(6)
    w = wl.scaled(wl.WORKLOADS[4], SCALED[5])
    check_case(gpu, rng, (w.modes_C, w.modes_A, w.modes_B),
               (w.shape("C"), w.shape("A"), w.shape("B")), dtype, 1.5, 0.5, flags=flags)


@pytest.mark.parametrize("dtype", DTYPES)
def test_unaligned_pointers_use_element_accesses(gpu, dtype):
    """Base pointers off the 16-byte grid: vector accesses must be dropped."""
    rng = np.random.default_rng(7)
    w = wl.scaled(wl.WORKLOADS[1], SCALED[2])
    check_case(gpu, rng, (w.modes_C, w.modes_A, w.modes_B),
               (w.shape("C"), w.shape("A"), w.shape("B")), dtype, 1.0, 1.0, offsets=(1, 3, 1))


@pytest.mark.parametrize("dtype", DTYPES)
def test_many_contracted_boxes(gpu, dtype):
    """Long contraction over several indices with ragged blocks."""
    rng = np.random.default_rng(8)
    modes = ("m,n", "k1,m,k2,k3", "k3,n,k2,k1")
    ext = {"m": 67, "n": 70, "k1": 13, "k2": 9, "k3": 21}
    shp = lambda s: [ext[x] for x in split(s)]
    check_case(gpu, rng, modes, (shp(modes[0]), shp(modes[1]), shp(modes[2])), dtype, 1.0, 0.0)


@pytest.mark.parametrize("dtype", DTYPES)
def test_zero_contracted_extent(gpu, dtype):
    rng = np.random.default_rng(9)
    C = make_operand(rng, [20, 30], dtype)
    A = make_operand(rng, [20, 0], dtype)
    B = make_operand(rng, [0, 30], dtype)
    ref = result_view(C.flat, C).astype(np.float64) * 0.5
    got_flat, _ = run_gpu(gpu, ("a,b", "a,k", "k,b"), (C, A, B), 1.0, 0.5)
    np.testing.assert_array_equal(result_view(got_flat, C).astype(np.float64), ref)


def test_plan_class_on_torch_views(gpu):
    import torch
    a = torch.randn(40, 30, 20, dtype=torch.float64, device=gpu).permute(2, 0, 1)  # (20,40,30)
    b = torch.randn(30, 50, dtype=torch.float64, device=gpu)
    c = torch.zeros(50, 20, 40, dtype=torch.float64, device=gpu)
    p = g.Plan("C[n,i,j] = A[i,j,k] * B[k,n]", C=c, A=a, B=b)
    p(a, b, c, 1.0, 0.0)
    torch.cuda.synchronize()
    ref = torch.einsum("ijk,kn->nij", a.cpu(), b.cpu())
    assert torch.allclose(c.cpu(), ref, rtol=1e-12, atol=1e-12)
    assert p.describe()["dtype"] == "f64"


TILES = {np.float32: 9, np.float64: 15}


@pytest.mark.parametrize("dtype,tile", [(dt, t) for dt in DTYPES for t in range(TILES[dt])])
@pytest.mark.parametrize("kind", [0, 1, 4])
@pytest.mark.parametrize("case", ["random", "smallk", "scaled2", "scaled3", "scaled4"])
def test_every_tile_shape(gpu, monkeypatch, dtype, tile, kind, case):
    """Each compiled tile shape and kernel kind (macro-kernel / persistent
    streaming kernel / direct-load kernel), forced through the analyser's
    test hooks (a kind the tile does not carry, or the plan cannot take,
    runs the tile's macro-kernel)."""
    monkeypatch.setenv("GETT_FORCE_TILE", str(tile))
    monkeypatch.setenv("GETT_FORCE_KIND", str(kind))
    rng = np.random.default_rng(30_000 + 10 * tile + kind)
    if case in ("random", "smallk"):
        while True:
            mc, ma, mb, ext = wl.random_problem(rng, max_rank=6, max_ext=9)
            kext = int(np.prod([ext[x] for x in split(ma) if x not in split(mc)]))
            if case == "random" or kext <= 16:
                break
        shp = lambda m: [ext[x] for x in split(m)]
        modes, shapes, alpha, beta = (mc, ma, mb), (shp(mc), shp(ma), shp(mb)), 1.5, -0.5
    else:
        w = wl.scaled(wl.WORKLOADS[int(case[-1]) - 1], SCALED[int(case[-1])])
        modes = (w.modes_C, w.modes_A, w.modes_B)
        shapes = (w.shape("C"), w.shape("A"), w.shape("B"))
        alpha, beta = w.alpha, w.beta
    check_case(gpu, rng, modes, shapes, dtype, alpha, beta)


@pytest.mark.parametrize("number", [2, 4])
def test_streaming_kernel_many_tiles_per_workgroup(gpu, monkeypatch, number):
    """The persistent streaming kernel with far more tiles than workgroups
    (each workgroup walks many tiles), at a size the oracle checks in full."""
    monkeypatch.setenv("GETT_FORCE_KIND", "1")
    big = {2: {"a": 128, "b": 100, "c": 64, "d": 20, "e": 16},
           4: {"a": 16, "b": 16, "c": 16, "d": 24, "i": 20, "j": 8, "k": 8}}[number]
    w = wl.scaled(wl.WORKLOADS[number - 1], big)
    rng = np.random.default_rng(w.seed + 7)
    check_case(gpu, rng, (w.modes_C, w.modes_A, w.modes_B),
               (w.shape("C"), w.shape("A"), w.shape("B")), w.np_dtype, w.alpha, w.beta)


@pytest.mark.parametrize("dtype,c_layout", [(np.float32, "col"), (np.float32, "row"),
                                            (np.float64, "col")])
def test_beyond_2_31_elements(gpu, dtype, c_layout):
    """C with 2^31 + 2^24 elements (8 GiB in fp32, 16 GiB in fp64): the tiles
    are reached through 64-bit base offsets (Sec. 2.2 allows tensors of any
    size).  C starts as NaN; every element is compared with the oracle.  With
    the row layout (n stride-one) the row offsets of C exceed 2^31 too."""
    import torch
    m, n, k = 65536, 32768 + 256, 8
    w = wl.Workload(900, "mn_2p31", "f32" if dtype == np.float32 else "f64", "m,n", "m,k",
                    "k,n", {"m": m, "n": n, "k": k})
    A, B, _ = wl.make_inputs(w)
    code = g.GETT_FLOAT32 if dtype == np.float32 else g.GETT_FLOAT64
    strides = None if c_layout == "col" else [n, 1]
    st, h = g.gett_plan(code, "m,n", [m, n], strides, "m,k", [m, k], None, "k,n", [k, n], None, 0)
    assert st == 0, g.gett_status_string(st)
    tA = torch.from_numpy(np.asfortranarray(A).reshape(-1, order="F")).to(gpu)
    tB = torch.from_numpy(np.asfortranarray(B).reshape(-1, order="F")).to(gpu)
    tdt = torch.float32 if dtype == np.float32 else torch.float64
    tC = torch.full((m * n,), float("nan"), dtype=tdt, device=gpu)
    try:
        st = g.gett_contract(h, 1.0, tA.data_ptr(), tB.data_ptr(), 0.0, tC.data_ptr(),
                             torch.cuda.current_stream().cuda_stream)
        assert st == 0
        torch.cuda.synchronize()
    finally:
        g.gett_destroy(h)
    assert bool(torch.isfinite(tC).all()), "some element of C was not written"
    if c_layout == "row":   # bring C to column-major order for the comparison
        tC = tC.view(m, n).t().contiguous().view(-1)
        torch.cuda.synchronize()
    err = compare_whole(tC, w, A, B, None, chunk=1 << 26)
    del tC
    torch.cuda.empty_cache()
    assert err <= TOL[dtype], f"rel err {err:.3e}"


@pytest.mark.parametrize("variant", ["8x8x8", "15x1x1"])
@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("kinds", [("dense",) * 3, ("permuted", "gapped", "permuted")])
def test_rank16(gpu, variant, dtype, kinds):
    """Tensors of 16 modes, every index kept by the plan, against the oracle
    (dense and permuted / gapped layouts; with permuted layouts some indices
    may merge)."""
    mc, ma, mb, ext = wl.rank16_problem(variant)
    rng = np.random.default_rng(90_000 + len(mc))
    shp = lambda m: [ext[x] for x in split(m)]
    check_case(gpu, rng, (mc, ma, mb), (shp(mc), shp(ma), shp(mb)), dtype, -0.75, 1.5, kinds)
