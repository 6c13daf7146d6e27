"""Plans of the direct-load kernels (no GPU needed): which plans the model
gives them, the fall-back to the tile's macro-kernel when the final gather
modes are not both vectors (or, for the persistent kernel, the contracted
set takes more than one box), and the K block lengths along an index that
vector gathers run along."""
import json

import pytest

import paper_1607_00145_amd as g
import workloads as wl
from gpu_util import split
from workloads import appendix_a as ap

DIRECT_TILES = {4, 7, 8}   # fp32 tiles that carry the direct-load kernel (none in fp64)


def describe(modes, ext, dtype=g.GETT_FLOAT32, strides=(None, None, None)):
    sh = [[ext[x] for x in split(m)] for m in modes]
    st, h = g.gett_plan(dtype, modes[0], sh[0], strides[0], modes[1], sh[1], strides[1],
                        modes[2], sh[2], strides[2], 0)
    assert st == 0
    try:
        return json.loads(g.gett_plan_describe(h))
    finally:
        g.gett_destroy(h)


def test_compute_bound_workload_is_direct():
    w = wl.BY_NAME["gemm4_fp32"]
    d = describe((w.modes_C, w.modes_A, w.modes_B), w.extents)
    assert d["kernel"] == "direct" and (d["tile"]["mt"], d["tile"]["nt"]) == (128, 256)
    assert d["partials"] == "none" and d["kslices"] == 1


def test_direct_candidates_only_on_tiles_that_carry_it():
    d = describe(("a,b", "a,k", "k,b"), {"a": 1024, "b": 1024, "k": 1024})
    kinds = {(c["tile"], c["kind"]) for c in d["candidates"]}
    assert {t for t, k in kinds if k == "direct"} == DIRECT_TILES
    d64 = describe(("a,b", "a,k", "k,b"), {"a": 1024, "b": 1024, "k": 1024}, g.GETT_FLOAT64)
    assert all(c["kind"] != "direct" for c in d64["candidates"])


def test_forced_direct_falls_back_without_vector_gathers(monkeypatch):
    """C's stride-one index a leads neither operand: the row operand is
    gathered element-wise, so the plan runs the macro-kernel."""
    monkeypatch.setenv("GETT_FORCE_TILE", "7")
    monkeypatch.setenv("GETT_FORCE_KIND", "4")
    d = describe(("a,b", "k,a", "k,b"), {"a": 512, "b": 512, "k": 64},
                 strides=(None, [512 * 64 + 1, 1], None))
    assert "scalar" in (d["gather_x"], d["gather_y"])
    assert d["kernel"] == "macro"
    d = describe(("a,b", "k,a", "k,b"), {"a": 512, "b": 512, "k": 64})
    assert d["kernel"] == "direct"


@pytest.mark.parametrize("k,tj,blocks", [(92, 32, 3), (104, 32, 4), (76, 32, 3), (96, 32, 3),
                                         (100, 20, 5), (48, 24, 2)])
def test_vector_index_block_length(k, tj, blocks):
    """Along the contracted index that k-vector gathers run along, a block
    length that divides the extent is taken unless it loses more than half of
    the box; otherwise the last block is ragged."""
    d = describe(("a,b", "a,k", "k,b"), {"a": 300, "b": 200, "k": k})
    assert d["gather_x"] == "k-vector" or d["gather_y"] == "k-vector"
    assert (d["kbox"]["tj"], d["kbox"]["blocks"]) == (tj, blocks)


def test_write_only_6d_workload_runs_the_persistent_kernel():
    w = wl.BY_NAME["ccsdt6_fp64"]
    d = describe((w.modes_C, w.modes_A, w.modes_B), w.extents, g.GETT_FLOAT64)
    assert d["kernel"] == "direct-stream" and d["kbox"]["steps"] == 1
    assert (d["tile"]["mt"], d["tile"]["nt"], d["tile"]["kt"]) == (64, 128, 24)


def test_persistent_candidates_only_on_the_fp64_one_box_tile():
    d = describe(("a,b", "a,k", "k,b"), {"a": 4096, "b": 4096, "k": 24}, g.GETT_FLOAT64)
    assert {c["tile"] for c in d["candidates"] if c["kind"] == "direct-stream"} == {14}
    d = describe(("a,b", "a,k", "k,b"), {"a": 4096, "b": 4096, "k": 16})
    assert all(c["kind"] != "direct-stream" for c in d["candidates"])
    # two K boxes: no candidate
    d = describe(("a,b", "a,k", "k,b"), {"a": 4096, "b": 4096, "k": 48}, g.GETT_FLOAT64)
    assert all(c["kind"] != "direct-stream" for c in d["candidates"])


@pytest.mark.parametrize("prefix,kernel", [("appA33_", "direct-stream"), ("appA46_", "direct-stream"),
                                           ("appA32_", "macro"), ("appA47_", "macro")])
def test_persistent_kernel_needs_long_c_runs(prefix, kernel):
    """6D contractions of Appendix A: a y set led by the merged run (a,b) of
    384 takes the persistent kernel; one led by a single index of 24 (C runs
    of 192 bytes) keeps the macro-kernel, which measured faster there."""
    w = next(x for x in ap.appendix_workloads("f64") if x.name.startswith(prefix))
    d = describe((w.modes_C, w.modes_A, w.modes_B), w.extents, g.GETT_FLOAT64)
    assert d["kernel"] == kernel, (w.name, d["y_order"])


def test_forced_persistent_kernel_falls_back(monkeypatch):
    """Forced onto a contracted set of two boxes, or onto an element-wise
    gather, the plan runs the tile's macro-kernel."""
    monkeypatch.setenv("GETT_FORCE_TILE", "14")
    monkeypatch.setenv("GETT_FORCE_KIND", "5")
    d = describe(("a,b", "a,k", "k,b"), {"a": 512, "b": 512, "k": 48}, g.GETT_FLOAT64)
    assert d["kernel"] == "macro"
    d = describe(("a,b", "k,a", "k,b"), {"a": 512, "b": 512, "k": 24}, g.GETT_FLOAT64,
                 strides=(None, [512 * 24 + 1, 1], None))
    assert "scalar" in (d["gather_x"], d["gather_y"]) and d["kernel"] == "macro"
    d = describe(("a,b", "k,a", "k,b"), {"a": 512, "b": 512, "k": 24}, g.GETT_FLOAT64)
    assert d["kernel"] == "direct-stream"
