"""Analyser decisions for K slices (host only): taken for small outputs with
long contracted sets, never for the benchmark workloads, never with the
deterministic flag, and reported in the plan's description."""
import json

import numpy as np
import pytest

import paper_1607_00145_amd as g
import workloads as wl
from workloads.appendix_a import appendix_workloads


def describe(w, flags=0):
    dt = g.GETT_FLOAT32 if w.dtype == "f32" else g.GETT_FLOAT64
    st, h = g.gett_plan(dt, w.modes_C, w.shape("C"), None, w.modes_A, w.shape("A"), None,
                        w.modes_B, w.shape("B"), None, flags)
    assert st == 0
    try:
        return json.loads(g.gett_plan_describe(h))
    finally:
        g.gett_destroy(h)


def test_workloads_are_not_sliced():
    for w in wl.WORKLOADS:
        d = describe(w)
        assert d["kslices"] == 1, w.name


@pytest.mark.parametrize("dtype", ["f32", "f64"])
def test_small_output_deep_k_is_sliced(dtype):
    """Appendix A's ab-acd-dbc and ab-cad-dcb: a C of about 1e5 elements over
    a contracted set of about 1e5: a few tiles, thousands of K boxes."""
    ws = {w.name.split("_")[1]: w for w in appendix_workloads(dtype)}
    for name in ("ab-acd-dbc", "ab-cad-dcb"):
        d = describe(ws[name])
        assert d["kslices"] >= 8, name
        assert d["grid"]["workgroups"] * d["kslices"] >= 256
        assert d["kbox"]["steps"] // d["kslices"] >= 8
        kinds = [c["kind"] for c in d["candidates"]]
        assert kinds[0] == "kslices"
        assert all(c["kslices"] > 1 for c in d["candidates"] if c["kind"] == "kslices")
        det = describe(ws[name], g.GETT_FLAG_DETERMINISTIC)
        assert det["kslices"] == 1
        assert all(c["kind"] != "kslices" for c in det["candidates"])


def test_force_hook(monkeypatch):
    w = wl.WORKLOADS[4]
    monkeypatch.setenv("GETT_FORCE_KSLICES", "6")
    assert describe(w)["kslices"] == 6
    assert describe(w, g.GETT_FLAG_DETERMINISTIC)["kslices"] == 1
    wa = [x for x in appendix_workloads("f64") if "ab-acd-dbc" in x.name][0]
    monkeypatch.setenv("GETT_FORCE_KSLICES", "1")
    assert describe(wa)["kslices"] == 1


def test_single_box_and_empty_cases_are_not_sliced():
    # one K box: nothing to share
    d = describe(wl.WORKLOADS[1])
    assert d["kbox"]["steps"] == 1 and d["kslices"] == 1
    # empty C and empty sums plan no slices
    st, h = g.gett_plan(g.GETT_FLOAT32, "m,n", [0, 5], None, "m,k", [0, 4000], None, "k,n",
                        [4000, 5], None, 0)
    assert st == 0
    assert json.loads(g.gett_plan_describe(h))["kslices"] == 1
    g.gett_destroy(h)


def test_slice_workspace_layout(monkeypatch):
    """K slices sum through the workspace: one counter per tile, one slot per
    (slice, tile) -- slot p * tiles + u for slice p of tile u, distinct by
    construction -- sized tiles x slices tile-sized slots."""
    w = wl.WORKLOADS[4]
    monkeypatch.setenv("GETT_FORCE_KSLICES", "6")
    d = describe(w)
    tiles = d["grid"]["workgroups"]
    tile_bytes = d["tile"]["mt"] * d["tile"]["nt"] * 4
    assert d["partials"] == "workspace"
    assert d["workspace_counters"] == tiles
    assert d["workspace_bytes"] == 6 * tiles * tile_bytes
    slots = {p * tiles + u for p in range(6) for u in range(tiles)}
    assert len(slots) == 6 * tiles and max(slots) < 6 * tiles
    monkeypatch.setenv("GETT_FORCE_KSLICES", "1")
    n = describe(w)
    assert n["partials"] == "none" and n["workspace_bytes"] == 0
