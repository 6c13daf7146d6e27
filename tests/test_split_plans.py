"""Analyser decisions for split index orders (Sec. 3.2.1, Fig. 5 and Examples
1-2): where a block of one stride-one index is placed before another, the
block sizes the kernels rely on, and where the split is refused.  Host
only."""
import json

import numpy as np
import pytest

import paper_1607_00145_amd as g
from test_gpu_split import CASES, COLUMN, EXPECT, FORCED, KSPLIT, TILES, describe, shapes_of

VW = {np.float32: 4, np.float64: 2}


def check_invariants(d, dtype, name):
    vw = VW[dtype]
    es = d["y_vector_stride"]
    if d["gather_y"] == "row-vector-strided":
        first = d["y_order"][0]
        assert first.endswith(f"<{es}") or es == 1
        assert d["tile"]["nt"] % (es * vw) == 0
        assert es >= vw and es & (es - 1) == 0
    elif d["gather_y"] == "k-vector-strided":
        assert d["k_order"][0].endswith(f"<{es}")
        assert d["tile"]["kt"] % (es * vw) == 0
        kb = d["kbox"]
        assert kb["kj"] >= 1
        if kb["kj"] == 1:
            assert kb["tj"] % vw == 0
        assert kb["elements"] <= d["tile"]["kt"]
        assert es >= vw and es & (es - 1) == 0
    else:
        assert es == 1


@pytest.mark.parametrize("dtype", [np.float32, np.float64])
@pytest.mark.parametrize("name", list(CASES))
def test_default_plans_split(name, dtype):
    modes, ext = CASES[name]
    d = describe(modes, ext, dtype)
    assert d["gather_y"] == EXPECT[name]
    check_invariants(d, dtype, name)
    if name in KSPLIT:
        # the row operand reads vectors along the block of its stride-one index
        assert d["gather_x"] == "k-vector"
    for flags in (g.GETT_FLAG_NO_SPLIT, g.GETT_FLAG_SCALAR):
        d = describe(modes, ext, dtype, flags)
        assert d["y_vector_stride"] == 1
        assert not any("<" in n for n in d["y_order"] + d["k_order"])


@pytest.mark.parametrize("dtype", [np.float32, np.float64])
@pytest.mark.parametrize("name", list(FORCED))
def test_forced_split_plan(monkeypatch, name, dtype):
    monkeypatch.setenv("GETT_SPLIT_F", str(FORCED[name]))
    modes, ext = CASES[name]
    d = describe(modes, ext, dtype)
    assert d["gather_y"] == "row-vector-strided"
    assert d["y_vector_stride"] == FORCED[name]
    check_invariants(d, dtype, name)


@pytest.mark.parametrize("dtype", [np.float32, np.float64])
@pytest.mark.parametrize("name", list(CASES))
def test_every_tile_keeps_the_invariants(monkeypatch, name, dtype):
    modes, ext = CASES[name]
    for tile in range(TILES[dtype]):
        for kind in (0, 1):
            monkeypatch.setenv("GETT_FORCE_TILE", str(tile))
            monkeypatch.setenv("GETT_FORCE_KIND", str(kind))
            d = describe(modes, ext, dtype)
            assert d["tile"]["id"] == tile
            check_invariants(d, dtype, name)
            if d["kernel"] == "stream":
                assert d["kbox"]["steps"] <= 1


def test_split_refused_where_it_cannot_hold():
    modes, ext = COLUMN["abc-bda-dc"]
    # C's stride-one extent odd: no block of it holds a vector
    d = describe(modes, {**ext, "a": 45}, np.float32)
    assert d["gather_y"] == "scalar"
    # the operand's stride-one extent not a multiple of the vector width
    d = describe(modes, {**ext, "b": 19}, np.float32)
    assert d["gather_y"] == "scalar"
    modes, ext = KSPLIT["abcd-eafb-fdec"]
    d = describe(modes, {**ext, "e": 23}, np.float32)      # B's... A's stride-one extent odd
    assert d["gather_y"] != "k-vector-strided"


def test_split_refused_for_misaligned_strides():
    """A split whose vectors would leave the 16-byte grid is not taken."""
    modes, ext = COLUMN["abc-bda-dc"]
    sh = shapes_of(modes, ext)
    # A[b,d,a] with d padded to an odd stride: rows of A start off the grid
    sA = [1, sh[1][0] + 1, (sh[1][0] + 1) * sh[1][1]]
    st, h = g.gett_plan(g.GETT_FLOAT32, modes[0], sh[0], None, modes[1], sh[1], sA,
                        modes[2], sh[2], None, 0)
    assert st == 0
    d = json.loads(g.gett_plan_describe(h))
    g.gett_destroy(h)
    assert d["gather_y"] == "scalar"
