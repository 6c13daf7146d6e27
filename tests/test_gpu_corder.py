"""GPU parity of the C-order epilogue: when C's stride-one run along the
tile's columns is shorter than a cache line and C continues in memory along
a row index, the runs wholly inside a tile are staged in LDS and stored in
C's memory order; runs cut by the tile's edges are stored per lane.  Against
the oracle for the index patterns of Appendix A's 6D contractions at reduced
extents (short runs kept, every other extent ragged), every beta path, and
bit for bit against the per-lane stores of the same plan."""
import json
import os

import numpy as np
import pytest

import paper_1607_00145_amd as g
from gpu_util import split
from test_gpu_parity import TILES, check_case

pytestmark = pytest.mark.gpu

# Appendix A rows 31, 32, 35 (C's a in one operand, b in the other)
PATTERNS = {
    "abcdef-dega-gfbc": ("a,b,c,d,e,f", "d,e,g,a", "g,f,b,c"),
    "abcdef-degb-gfac": ("a,b,c,d,e,f", "d,e,g,b", "g,f,a,c"),
    "abcdef-dfgb-geac": ("a,b,c,d,e,f", "d,f,g,b", "g,e,a,c"),
}
EXT = {np.float32: {"a": 24, "b": 7, "c": 5, "d": 9, "e": 4, "f": 3, "g": 12},
       np.float64: {"a": 8, "b": 11, "c": 5, "d": 9, "e": 4, "f": 3, "g": 10}}
# the tiles the paper-size plans of these contractions use
TILE = {np.float32: "3", np.float64: "11"}


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


@pytest.mark.parametrize("dtype", [np.float32, np.float64])
@pytest.mark.parametrize("name", list(PATTERNS))
def test_c_order_against_oracle(gpu, monkeypatch, name, dtype):
    """fp32 tiles carry the C-order epilogue; fp64 plans of the same
    patterns keep the per-lane stores (and their element-wise gathers the
    lane order)."""
    monkeypatch.setenv("GETT_FORCE_TILE", TILE[dtype])
    monkeypatch.setenv("GETT_FORCE_KIND", "0")
    modes, ext = PATTERNS[name], EXT[dtype]
    d = describe(modes, ext, dtype)
    assert d["c_order_run"] == (ext["a"] if dtype == np.float32 else 0)
    rng = np.random.default_rng(sum(map(ord, name)))
    for alpha, beta in [(1.0, 0.0), (-1.5, 0.5), (2.0, 1.0), (0.0, -1.0)]:
        check_case(gpu, rng, modes, shapes(modes, ext), dtype, alpha, beta)
    # gapped / permuted operands (C dense keeps the short run)
    check_case(gpu, rng, modes, shapes(modes, ext), dtype, 0.75, -0.25,
               kinds=("dense", "gapped", "permuted"))
    got, ref = check_case(gpu, rng, modes, shapes(modes, ext), dtype, 1.0, 1.0, dist="int")
    np.testing.assert_array_equal(got.astype(np.float64), ref.out64)


@pytest.mark.parametrize("dtype", [np.float32])
@pytest.mark.parametrize("name", list(PATTERNS))
def test_c_order_same_bits_as_per_lane(gpu, monkeypatch, name, dtype):
    """The staged stores compute alpha * acc + beta * C exactly as the
    per-lane stores do: identical bits."""
    monkeypatch.setenv("GETT_FORCE_TILE", TILE[dtype])
    monkeypatch.setenv("GETT_FORCE_KIND", "0")
    modes, ext = PATTERNS[name], EXT[dtype]
    outs = []
    for co in ("1", "0"):
        monkeypatch.setenv("GETT_C_ORDER", co)
        assert (describe(modes, ext, dtype)["c_order_run"] > 0) == (co == "1")
        rng = np.random.default_rng(4)
        got, _ = check_case(gpu, rng, modes, shapes(modes, ext), dtype, 1.25, -0.75)
        outs.append(got.copy())
    np.testing.assert_array_equal(outs[0], outs[1])


@pytest.mark.parametrize("dtype,tile", [(dt, t) for dt in (np.float32, np.float64)
                                        for t in range(TILES[dt])])
def test_c_order_every_tile(gpu, monkeypatch, dtype, tile):
    monkeypatch.setenv("GETT_FORCE_TILE", str(tile))
    monkeypatch.setenv("GETT_FORCE_KIND", "0")
    modes, ext = PATTERNS["abcdef-dega-gfbc"], EXT[dtype]
    rng = np.random.default_rng(600 + tile)
    check_case(gpu, rng, modes, shapes(modes, ext), dtype, 1.5, 0.5)
    check_case(gpu, rng, modes, shapes(modes, ext), dtype, 1.0, 0.0)


@pytest.mark.parametrize("dtype", [np.float32, np.float64])
@pytest.mark.parametrize("name", list(PATTERNS))
def test_lane_order_same_bits(gpu, monkeypatch, name, dtype):
    """Element-wise gathers walking the operand's stride-one index (rows
    grouped by the first index's value) pack the same tiles: identical bits
    with and without the lane order."""
    monkeypatch.setenv("GETT_FORCE_TILE", TILE[dtype])
    monkeypatch.setenv("GETT_FORCE_KIND", "0")
    modes, ext = PATTERNS[name], EXT[dtype]
    if max(describe(modes, ext, dtype)["lane_perm"]) == 0:
        pytest.skip("this plan gathers both operands in vectors")
    outs = []
    for lp in ("1", "0"):
        monkeypatch.setenv("GETT_LANE_PERM", lp)
        d = describe(modes, ext, dtype)
        assert (max(d["lane_perm"]) > 0) == (lp == "1")
        rng = np.random.default_rng(8)
        got, _ = check_case(gpu, rng, modes, shapes(modes, ext), dtype, -1.0, 0.5)
        outs.append(got.copy())
    np.testing.assert_array_equal(outs[0], outs[1])
