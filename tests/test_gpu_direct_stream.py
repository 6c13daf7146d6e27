"""GPU parity of the persistent direct-load kernel (plans whose contracted set
is one K box; fp64 tile 64 x 128 x 24): every pair of vector gather modes, a
whole box, a partial box and a short one, workgroups that walk several tiles
(more tiles than resident workgroups), ragged tiles, the 6D x 4D structure of
the write-only fp64 workload, every beta path, integer inputs (exact whatever
the order of the additions), C unaligned or gapped (single-element stores),
and the calls that run the tile's macro-kernel instead (alpha = 0, operands
not 16-byte aligned, a contracted set of two boxes), against the oracle."""
import json

import numpy as np
import pytest

import paper_1607_00145_amd as g
from gpu_util import split
from test_gpu_parity import check_case

pytestmark = pytest.mark.gpu
TILE = "14"   # fp64 64 x 128 x 24, one K box

MODE_CASES = {
    "ab-ak-kb": (("a,b", "a,k", "k,b"), ("k-vector", "row-vector")),
    "ab-ka-kb": (("a,b", "k,a", "k,b"), ("k-vector", "k-vector")),
    "ab-ak-bk": (("a,b", "a,k", "b,k"), ("row-vector", "row-vector")),
    "ab-ka-bk": (("a,b", "k,a", "b,k"), ("row-vector", "k-vector")),
    "ba-ak-kb": (("b,a", "a,k", "k,b"), ("row-vector", "k-vector")),
}


def shapes(modes, ext):
    return tuple([ext[x] for x in split(m)] for m in modes)


def describe(modes, ext):
    sh = shapes(modes, ext)
    st, h = g.gett_plan(g.GETT_FLOAT64, modes[0], sh[0], None, modes[1], sh[1], None, modes[2],
                        sh[2], None, 0)
    assert st == 0
    try:
        return json.loads(g.gett_plan_describe(h))
    finally:
        g.gett_destroy(h)


@pytest.fixture
def forced(monkeypatch):
    monkeypatch.setenv("GETT_FORCE_TILE", TILE)
    monkeypatch.setenv("GETT_FORCE_KIND", "5")


@pytest.mark.parametrize("k", [24, 20, 8])
@pytest.mark.parametrize("name", list(MODE_CASES))
def test_direct_stream_gather_modes(gpu, forced, name, k):
    modes, (gx, gy) = MODE_CASES[name]
    ext = {"a": 768, "b": 512, "k": k}
    d = describe(modes, ext)
    assert d["kernel"] == "direct-stream" and d["tile"]["id"] == int(TILE)
    assert (d["gather_x"], d["gather_y"]) == (gx, gy)
    assert d["kbox"]["steps"] == 1
    rng = np.random.default_rng(2000 + 10 * k + len(name))
    for alpha, beta in [(1.0, 0.0), (-0.75, 1.0), (1.5, -0.5)]:
        check_case(gpu, rng, modes, shapes(modes, ext), np.float64, alpha, beta)


@pytest.mark.parametrize("name", ["ab-ak-kb", "ab-ka-bk"])
def test_direct_stream_walks_several_tiles(gpu, forced, name):
    """4096 x 2048 of 64 x 128 tiles: 1024 tiles, more than the resident
    workgroups, so each walks two or more; integer inputs, compared exactly."""
    modes = MODE_CASES[name][0]
    ext = {"a": 4096, "b": 2048, "k": 24}
    assert describe(modes, ext)["kernel"] == "direct-stream"
    rng = np.random.default_rng(31 + len(name))
    for beta in (0.0, 2.0):
        got, ref = check_case(gpu, rng, modes, shapes(modes, ext), np.float64, 1.0, beta,
                              dist="int")
        np.testing.assert_array_equal(got.astype(np.float64), ref.out64)


RAGGED = {
    "ab-ak-kb": (("a,b", "a,k", "k,b"), {"a": 300, "b": 200, "k": 24}),
    "ab-ka-kb": (("a,b", "k,a", "k,b"), {"a": 2000, "b": 136, "k": 22}),
    "ab-ak-bk": (("a,b", "a,k", "b,k"), {"a": 140, "b": 3000, "k": 6}),
    "abcijk-dabi-cdjk": (("a,b,c,i,j,k", "d,a,b,i", "c,d,j,k"),
                         {"a": 8, "b": 8, "c": 8, "i": 8, "j": 8, "k": 6, "d": 24}),
    "abcijk-dabi-cdjk-r": (("a,b,c,i,j,k", "d,a,b,i", "c,d,j,k"),
                           {"a": 6, "b": 10, "c": 10, "i": 9, "j": 4, "k": 10, "d": 14}),
}


@pytest.mark.parametrize("name", list(RAGGED))
def test_direct_stream_ragged_and_6d(gpu, forced, name):
    modes, ext = RAGGED[name]
    d = describe(modes, ext)
    assert d["kernel"] == "direct-stream"
    rng = np.random.default_rng(700 + len(name))
    for alpha, beta in [(1.0, 0.0), (-0.5, 1.5)]:
        check_case(gpu, rng, modes, shapes(modes, ext), np.float64, alpha, beta)
    got, ref = check_case(gpu, rng, modes, shapes(modes, ext), np.float64, 1.0, 1.0, dist="int")
    np.testing.assert_array_equal(got.astype(np.float64), ref.out64)


def test_direct_stream_fallbacks(gpu, forced):
    """alpha = 0 (C <- beta C), operands whose base is not 16-byte aligned and
    a contracted set of two boxes run the tile's macro-kernel."""
    modes = MODE_CASES["ab-ak-kb"][0]
    ext = {"a": 256, "b": 256, "k": 24}
    rng = np.random.default_rng(5)
    for beta in (0.0, -1.5):
        check_case(gpu, rng, modes, shapes(modes, ext), np.float64, 0.0, beta)
    for offsets in [(0, 1, 0), (0, 0, 1), (1, 3, 1)]:
        check_case(gpu, rng, modes, shapes(modes, ext), np.float64, 1.0, 0.5, offsets=offsets)
    ext2 = {"a": 256, "b": 256, "k": 48}
    assert describe(modes, ext2)["kernel"] == "macro"
    check_case(gpu, rng, modes, shapes(modes, ext2), np.float64, 1.0, 0.5)


@pytest.mark.parametrize("beta", [0.0, 1.5])
def test_direct_stream_unaligned_or_gapped_c(gpu, forced, beta):
    """C whose base is not 16-byte aligned, or C with gaps between its rows:
    the persistent kernel still runs (its operands are aligned) and stores
    single elements (whole tiles: every store issued, no offset checks)."""
    modes = MODE_CASES["ab-ak-kb"][0]
    ext = {"a": 1024, "b": 768, "k": 24}
    assert describe(modes, ext)["kernel"] == "direct-stream"
    rng = np.random.default_rng(77)
    check_case(gpu, rng, modes, shapes(modes, ext), np.float64, 1.0, beta, offsets=(1, 0, 0))
    check_case(gpu, rng, modes, shapes(modes, ext), np.float64, -0.5, beta,
               kinds=("gapped", "dense", "dense"))
    got, ref = check_case(gpu, rng, modes, shapes(modes, ext), np.float64, 1.0, beta,
                          dist="int", offsets=(1, 0, 0))
    np.testing.assert_array_equal(got.astype(np.float64), ref.out64)
