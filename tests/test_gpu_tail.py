"""GPU parity of the stream-K tail: whole tiles for the complete rounds of
workgroups, and the K boxes of the remaining tiles dealt in equal runs to
further workgroups whose partial tiles are summed in piece order through the
library's workspace.  Against the oracle with the tail
kernel forced on tiles that carry it and the tail spread over a chosen number
of workgroups (runs that end inside a tile, runs that cover several tiles,
one workgroup for all of it), every beta path, alpha = 0, integer inputs
(exact whatever the order of the additions), permuted and gapped layouts, and
the model's own choice at the extents of the 4D x 4D fp64 workload."""
import json

import numpy as np
import pytest

import paper_1607_00145_amd as g
from gpu_util import split
from test_gpu_parity import check_case

pytestmark = pytest.mark.gpu
TAIL_TILE = {np.float32: "2", np.float64: "8"}
DTYPES = [np.float32, np.float64]

# several tiles along both free sets (ragged), deep contracted sets
CASES = {
    "abij-iejf-faeb": (("a,b,i,j", "i,e,j,f", "f,a,e,b"),
                       {"a": 23, "b": 17, "i": 19, "j": 21, "e": 13, "f": 11}),
    "ab-ak-kb": (("a,b", "a,k", "k,b"), {"a": 300, "b": 290, "k": 333}),
    "abc-adc-db": (("a,b,c", "a,d,c", "d,b"), {"a": 45, "b": 200, "c": 7, "d": 150}),
    # one K box: every tail run is whole tiles
    "abcd-aeb-edc": (("a,b,c,d", "a,e,b", "e,d,c"), {"a": 30, "b": 17, "c": 29, "d": 31, "e": 16}),
}


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


def force_tail(monkeypatch, dtype, wgs):
    monkeypatch.setenv("GETT_FORCE_TILE", TAIL_TILE[dtype])
    monkeypatch.setenv("GETT_FORCE_KIND", "3")
    monkeypatch.setenv("GETT_TAIL_WGS", str(wgs))


def check_cover(d):
    """The tail workgroups' runs cover the boxes of every tile after the
    whole ones."""
    t = d["tail"]
    tiles = d["grid"]["tiles_x"] * d["grid"]["tiles_y"]
    assert d["kernel"] == "tail"
    assert 0 <= t["full_tiles"] < tiles and t["workgroups"] >= 1
    boxes = (tiles - t["full_tiles"]) * d["kbox"]["steps"]
    assert t["workgroups"] * t["boxes"] >= boxes > (t["workgroups"] - 1) * t["boxes"]


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("wgs", [1, 3, 7, 40, 256])
@pytest.mark.parametrize("name", list(CASES))
def test_forced_tail(gpu, monkeypatch, name, wgs, dtype):
    force_tail(monkeypatch, dtype, wgs)
    modes, ext = CASES[name]
    d = describe(modes, ext, dtype)
    check_cover(d)
    assert d["partials"] == "workspace"
    rng = np.random.default_rng(100 * wgs + len(name))
    for alpha, beta in [(1.0, 0.0), (-0.75, 1.0), (1.5, -0.5)]:
        check_case(gpu, rng, modes, shapes(modes, ext), dtype, alpha, beta)


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("name", list(CASES))
def test_tail_integer_inputs_exact(gpu, monkeypatch, name, dtype):
    force_tail(monkeypatch, dtype, 5)
    modes, ext = CASES[name]
    rng = np.random.default_rng(33)
    for beta in (0.0, 1.0, 2.0):
        got, ref = check_case(gpu, rng, modes, shapes(modes, ext), dtype, 1.0, beta, dist="int")
        np.testing.assert_array_equal(got.astype(np.float64), ref.out64)


@pytest.mark.parametrize("dtype", DTYPES)
def test_tail_layouts_and_alpha_zero(gpu, monkeypatch, dtype):
    force_tail(monkeypatch, dtype, 6)
    modes, ext = CASES["abij-iejf-faeb"]
    rng = np.random.default_rng(71)
    for kinds in [("gapped",) * 3, ("permuted", "gapped", "dense"), ("dense", "permuted", "permuted")]:
        check_case(gpu, rng, modes, shapes(modes, ext), dtype, 0.5, 0.25, kinds=kinds)
    for beta in (0.0, -1.5):
        check_case(gpu, rng, modes, shapes(modes, ext), dtype, 0.0, beta)


@pytest.mark.parametrize("dtype", DTYPES)
def test_tail_not_with_deterministic_flag(gpu, monkeypatch, dtype):
    force_tail(monkeypatch, dtype, 4)
    modes, ext = CASES["ab-ak-kb"]
    assert describe(modes, ext, dtype, g.GETT_FLAG_DETERMINISTIC)["kernel"] == "macro"
    rng = np.random.default_rng(5)
    check_case(gpu, rng, modes, shapes(modes, ext), dtype, 1.0, 0.5,
               flags=g.GETT_FLAG_DETERMINISTIC)
