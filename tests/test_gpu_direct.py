"""GPU parity of the direct-load kernel, whose operands are copied from device
memory straight into LDS (fp32 tiles 128 x 128 x 32, 256 x 128 x 32 and
128 x 256 x 32):
every pair of vector gather modes, one to five K boxes, boxes over two
contracted indices, ragged tiles and partial boxes (pieces outside the
tensors written as zeros; a partial last box reuses a buffer that held
another box), every beta path, alpha = 0, integer inputs (exact whatever the
order of the additions), and the calls that fall back to the macro-kernel
of the plan's tile (operands whose base is not 16-byte aligned, alpha = 0),
against the oracle."""
import json

import numpy as np
import pytest

import paper_1607_00145_amd as g
from gpu_util import split
from test_gpu_parity import check_case

pytestmark = pytest.mark.gpu
# (dtype, tile) pairs that carry the direct-load kernel
DIRECT_TILES = [(np.float32, "4"), (np.float32, "7"), (np.float32, "8")]
IDS = ["f32-4", "f32-7", "f32-8"]
BOX = {np.float32: 32, np.float64: 16}   # KT of those tiles

# name: (modes of C, A, B), gather modes (x, y) of the plan; the free extents
# are multiples of both tiles, K is set per test
MODE_CASES = {
    "ab-ak-kb": (("a,b", "a,k", "k,b"), ("k-vector", "row-vector")),
    "ab-ka-kb": (("a,b", "k,a", "k,b"), ("k-vector", "k-vector")),
    "ab-ak-bk": (("a,b", "a,k", "b,k"), ("row-vector", "row-vector")),
    "ab-ka-bk": (("a,b", "k,a", "b,k"), ("row-vector", "k-vector")),
    "ba-ak-kb": (("b,a", "a,k", "k,b"), ("row-vector", "k-vector")),
}


def shapes(modes, ext):
    return tuple([ext[x] for x in split(m)] for m in modes)


def describe(modes, ext, dtype=np.float32):
    sh = shapes(modes, ext)
    code = g.GETT_FLOAT32 if dtype == np.float32 else g.GETT_FLOAT64
    st, h = g.gett_plan(code, modes[0], sh[0], None, modes[1], sh[1], None, modes[2], sh[2], None,
                        0)
    assert st == 0
    try:
        return json.loads(g.gett_plan_describe(h))
    finally:
        g.gett_destroy(h)


def force_direct(monkeypatch, tile):
    monkeypatch.setenv("GETT_FORCE_TILE", tile)
    monkeypatch.setenv("GETT_FORCE_KIND", "4")


@pytest.mark.parametrize("k", [32, 64, 96, 160])
@pytest.mark.parametrize("name", list(MODE_CASES))
@pytest.mark.parametrize("dtype,tile", DIRECT_TILES, ids=IDS)
def test_direct_gather_modes(gpu, monkeypatch, dtype, tile, name, k):
    force_direct(monkeypatch, tile)
    modes, (gx, gy) = MODE_CASES[name]
    ext = {"a": 768, "b": 512, "k": k}
    d = describe(modes, ext, dtype)
    assert d["kernel"] == "direct" and d["tile"]["id"] == int(tile)
    assert (d["gather_x"], d["gather_y"]) == (gx, gy)
    assert d["kbox"]["steps"] == k // BOX[dtype]
    rng = np.random.default_rng(1000 * k + len(name) + int(tile))
    for alpha, beta in [(1.0, 0.0), (-0.75, 1.0), (1.5, -0.5)]:
        check_case(gpu, rng, modes, shapes(modes, ext), dtype, alpha, beta)


@pytest.mark.parametrize("dtype,tile", DIRECT_TILES, ids=IDS)
def test_direct_boxes_over_two_indices(gpu, monkeypatch, dtype, tile):
    """A box of k whole (8) and a block of l (extent 12): 4 of l per box in
    fp32 (three boxes), 2 in fp64 (six)."""
    force_direct(monkeypatch, tile)
    modes = ("a,b,c,d", "k,a,l,b", "c,l,d,k")
    ext = {"a": 16, "b": 16, "c": 32, "d": 8, "k": 8, "l": 12}
    d = describe(modes, ext, dtype)
    assert d["kernel"] == "direct"
    assert d["kbox"]["kj"] == 1 and d["kbox"]["elements"] == BOX[dtype]
    assert d["kbox"]["steps"] == 12 // (BOX[dtype] // 8)
    rng = np.random.default_rng(7)
    for alpha, beta in [(1.0, 0.0), (0.5, 2.0)]:
        check_case(gpu, rng, modes, shapes(modes, ext), dtype, alpha, beta)


@pytest.mark.parametrize("dtype,tile", DIRECT_TILES, ids=IDS)
def test_direct_integer_inputs_exact(gpu, monkeypatch, dtype, tile):
    force_direct(monkeypatch, tile)
    rng = np.random.default_rng(99)
    for name in ("ab-ak-kb", "ab-ka-bk"):
        modes = MODE_CASES[name][0]
        ext = {"a": 256, "b": 512, "k": 224}
        for beta in (0.0, 1.0, 2.0):
            got, ref = check_case(gpu, rng, modes, shapes(modes, ext), dtype, 1.0, beta,
                                  dist="int")
            np.testing.assert_array_equal(got.astype(np.float64), ref.out64)


@pytest.mark.parametrize("dtype,tile", DIRECT_TILES, ids=IDS)
def test_direct_alpha_zero_and_gemm4_structure(gpu, monkeypatch, dtype, tile):
    """alpha = 0 (C <- beta C, the macro-kernel of the tile) and the 4D x 4D
    index structure of the compute-bound fp32 workload at 256 x 256 x 512."""
    force_direct(monkeypatch, tile)
    modes = ("m1,n1,m2,n2", "m1,k1,m2,k2", "k2,n1,k1,n2")
    ext = {"m1": 64, "m2": 4, "n1": 64, "n2": 4, "k1": 8, "k2": 64}
    d = describe(modes, ext, dtype)
    assert d["kernel"] == "direct" and d["kbox"]["steps"] == 512 // BOX[dtype]
    rng = np.random.default_rng(3)
    check_case(gpu, rng, modes, shapes(modes, ext), dtype, -1.25, 0.5)
    for beta in (0.0, -1.5):
        check_case(gpu, rng, modes, shapes(modes, ext), dtype, 0.0, beta)


# ragged free extents (no multiple of either tile) and contracted sets whose
# boxes are partial: k = 104 (three boxes of 32 and one of 8, in a buffer
# that held box 1), k = 28 (one box of 28 positions), and a box over two
# indices whose last block is short (l = 10 in blocks of 4)
RAGGED = {
    "ab-ak-kb": (("a,b", "a,k", "k,b"), {"a": 300, "b": 200, "k": 104}),
    "ab-ka-kb": (("a,b", "k,a", "k,b"), {"a": 264, "b": 136, "k": 28}),
    "ab-ak-bk": (("a,b", "a,k", "b,k"), {"a": 140, "b": 388, "k": 104}),
    "ab-ka-bk": (("a,b", "k,a", "b,k"), {"a": 520, "b": 68, "k": 72}),
    "abcd-kalb-cldk": (("a,b,c,d", "k,a,l,b", "c,l,d,k"),
                       {"a": 12, "b": 20, "c": 36, "d": 5, "k": 8, "l": 10}),
}


@pytest.mark.parametrize("name", list(RAGGED))
@pytest.mark.parametrize("dtype,tile", DIRECT_TILES, ids=IDS)
def test_direct_ragged_tiles_and_partial_boxes(gpu, monkeypatch, dtype, tile, name):
    force_direct(monkeypatch, tile)
    modes, ext = RAGGED[name]
    d = describe(modes, ext, dtype)
    assert d["kernel"] == "direct"
    rng = np.random.default_rng(500 + len(name) + int(tile))
    for alpha, beta in [(1.0, 0.0), (-0.5, 1.5)]:
        check_case(gpu, rng, modes, shapes(modes, ext), dtype, alpha, beta)
    for beta in (0.0, 1.0):
        got, ref = check_case(gpu, rng, modes, shapes(modes, ext), dtype, 1.0, beta,
                              dist="int")
        np.testing.assert_array_equal(got.astype(np.float64), ref.out64)


@pytest.mark.parametrize("dtype,tile", DIRECT_TILES, ids=IDS)
def test_direct_fallbacks(gpu, monkeypatch, dtype, tile):
    """Operands whose base is not 16-byte aligned (their vector gathers
    become element-wise) run the macro-kernel of the direct plan's tile; so
    does a K box that two operands cannot both gather in vectors."""
    force_direct(monkeypatch, tile)
    modes = ("a,b,c", "a,k,l", "l,k,b,c")
    ext = {"a": 256, "b": 16, "c": 16, "k": 8, "l": 12}
    rng = np.random.default_rng(11)
    check_case(gpu, rng, modes, shapes(modes, ext), dtype, 1.0, 1.0)
    modes = MODE_CASES["ab-ak-kb"][0]
    ext = {"a": 256, "b": 256, "k": 64}
    assert describe(modes, ext, dtype)["kernel"] == "direct"
    for offsets in [(0, 1, 0), (0, 0, 1), (1, 3, 1)]:
        check_case(gpu, rng, modes, shapes(modes, ext), dtype, 1.0, 0.5, offsets=offsets)
