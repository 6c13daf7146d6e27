"""Analyser decisions for the stream-K tail (host only): the split of the
tiles into whole ones and a tail, and the tail workgroups' runs of K boxes,
replayed on the CPU the way the kernel walks them: every box of every tail
tile is summed exactly once, every workgroup gets boxes, and no run reaches
past the last tile.  The deterministic flag and an empty C keep the plain
kernel."""
import json

import numpy as np
import pytest

import paper_1607_00145_amd as g
from gpu_util import split

TAIL_TILE = {"f32": "2", "f64": "8"}
SHAPES = {
    "abij-iejf-faeb": (("a,b,i,j", "i,e,j,f", "f,a,e,b"),
                       {"a": 23, "b": 17, "i": 19, "j": 21, "e": 13, "f": 11}),
    "ab-ak-kb": (("a,b", "a,k", "k,b"), {"a": 300, "b": 290, "k": 333}),
    "abc-adc-db": (("a,b,c", "a,d,c", "d,b"), {"a": 45, "b": 200, "c": 7, "d": 150}),
    # one K box: every tail run is whole tiles
    "abcd-aeb-edc": (("a,b,c,d", "a,e,b", "e,d,c"), {"a": 30, "b": 17, "c": 29, "d": 31, "e": 16}),
    "cc4x4": (("a,b,i,j", "i,e,j,f", "f,a,e,b"), {x: 48 for x in "abijef"}),
}


def describe(modes, ext, dtype, flags=0):
    code = g.GETT_FLOAT32 if dtype == "f32" else g.GETT_FLOAT64
    sh = tuple([ext[x] for x in split(m)] for m in modes)
    st, h = g.gett_plan(code, modes[0], sh[0], None, modes[1], sh[1], None, modes[2], sh[2],
                        None, flags)
    assert st == 0
    try:
        return json.loads(g.gett_plan_describe(h))
    finally:
        g.gett_destroy(h)


def walk(full, wgs, length, tiles, nb, slots_cap=None):
    """The tail kernel's decomposition: workgroup b < full takes tile b whole;
    workgroup full + j sums boxes [j * length, (j + 1) * length) of the
    concatenated box sequences of tiles full, full + 1, ...  A piece that is
    not a whole tile is saved in slot j + u (u: tail tile) and counted; the
    last of tile u's np pieces sums slots jf(u) + u + p, p = 0 .. np - 1,
    jf(u) = floor(u nb / length).  Checks that the slots are distinct and
    within the workspace the plan sizes, that each tile's pieces are exactly
    the slots its last piece sums, in run order."""
    count = np.zeros((tiles, nb), dtype=np.int64)
    count[:full] += 1
    total = (tiles - full) * nb
    saved = {}                          # slot -> (tail tile, run)
    pieces = {}                         # tail tile -> runs holding part of it
    for j in range(wgs):
        pos, end = j * length, min((j + 1) * length, total)
        assert pos < end, "a tail workgroup without boxes"
        while pos < end:
            u, s0 = divmod(pos, nb)
            n = min(nb - s0, end - pos)
            assert full + u < tiles
            count[full + u, s0:s0 + n] += 1
            if n < nb:
                jf, jl = u * nb // length, ((u + 1) * nb - 1) // length
                assert jf <= j <= jl
                slot = j + u
                assert slot not in saved, "two pieces in one slot"
                saved[slot] = (u, j)
                pieces.setdefault(u, []).append(j)
            pos += n
    r = tiles - full
    for u, runs in pieces.items():
        jf, jl = u * nb // length, ((u + 1) * nb - 1) // length
        assert runs == list(range(jf, jl + 1))                       # np = jl - jf + 1 pieces
        assert [saved[jf + u + p] for p in range(len(runs))] == [(u, x) for x in runs]
    if slots_cap is not None and saved:
        assert max(saved) < slots_cap == wgs + r - 1
    return count


@pytest.mark.parametrize("dtype", ["f32", "f64"])
@pytest.mark.parametrize("wgs", [1, 2, 3, 7, 40, 256, 100000])
@pytest.mark.parametrize("name", list(SHAPES))
def test_tail_covers_every_box_once(monkeypatch, name, wgs, dtype):
    monkeypatch.setenv("GETT_FORCE_TILE", TAIL_TILE[dtype])
    monkeypatch.setenv("GETT_FORCE_KIND", "3")
    monkeypatch.setenv("GETT_TAIL_WGS", str(wgs))
    d = describe(*SHAPES[name], dtype)
    assert d["kernel"] == "tail"
    t = d["tail"]
    tiles = d["grid"]["tiles_x"] * d["grid"]["tiles_y"]
    nb = d["kbox"]["steps"]
    rem = tiles % wgs or min(wgs, tiles)
    assert t["full_tiles"] == tiles - rem
    assert t["workgroups"] <= min(wgs, rem * nb)
    tile_bytes = d["tile"]["mt"] * d["tile"]["nt"] * (4 if dtype == "f32" else 8)
    assert d["partials"] == "workspace"
    assert d["workspace_counters"] == tiles - t["full_tiles"]
    assert d["workspace_bytes"] % tile_bytes == 0
    count = walk(t["full_tiles"], t["workgroups"], t["boxes"], tiles, nb,
                 slots_cap=d["workspace_bytes"] // tile_bytes)
    assert (count == 1).all()


@pytest.mark.parametrize("dtype", ["f32", "f64"])
def test_tail_not_deterministic_or_untiled(monkeypatch, dtype):
    monkeypatch.setenv("GETT_FORCE_TILE", TAIL_TILE[dtype])
    monkeypatch.setenv("GETT_FORCE_KIND", "3")
    modes, ext = SHAPES["ab-ak-kb"]
    d = describe(modes, ext, dtype, g.GETT_FLAG_DETERMINISTIC)
    assert d["kernel"] == "macro" and d["tail"]["workgroups"] == 0
    d = describe(modes, dict(ext, a=0), dtype)
    assert d["kernel"] == "macro"


def test_tail_only_on_tiles_that_carry_it(monkeypatch):
    """A tile compiled without the tail kernel is never given it."""
    monkeypatch.setenv("GETT_FORCE_TILE", "0")
    monkeypatch.setenv("GETT_FORCE_KIND", "3")
    d = describe(*SHAPES["ab-ak-kb"], "f64")
    assert d["kernel"] == "macro"
    for c in d["candidates"]:
        assert c["kind"] != "tail" or c["tile"] == 8
