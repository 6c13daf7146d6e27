"""The benchmark of Appendix A (Tables III and IV) on the host: the shapes as
transcribed obey the paper's own rules, every contraction plans, and the
Loops-over-GEMM applicability matches the paper's LoG column."""
import json

import pytest

import paper_1607_00145_amd as g
import workloads as wl
from workloads.appendix_a import TABLE, appendix_workloads, log_applicable


def test_table_is_well_formed():
    assert len(TABLE) == 48
    assert len({name for name, _, _, _ in TABLE}) == 48
    for name, sp, dp, _ in TABLE:
        c, a, b = name.split("-")
        idx = set(c) | set(a) | set(b)
        assert set(sp) == idx and set(dp) == idx, name
        for x in idx:   # every index in exactly two of the three tensors (Sec. 2.2, fn. 9)
            assert (x in c) + (x in a) + (x in b) == 2, (name, x)


@pytest.mark.parametrize("dtype,item", [("f32", 4), ("f64", 8)])
def test_sizing_rule(dtype, item):
    """Sec. 7.1: every test case is sized so that it needs at least 200 MiB
    (its largest tensor is at least that big), in both precisions."""
    for w in appendix_workloads(dtype):
        largest = max(w.numel(t) for t in "CAB") * item
        assert largest >= 200 * 2 ** 20, w.name


def test_log_applicability_matches_the_paper():
    """Listing 7's conditions, as implemented by gett_log_plan, refuse exactly
    the 15 contractions for which Tables III and IV report no LoG result."""
    paper = log_applicable()
    assert sum(not v for v in paper.values()) == 15
    for w in appendix_workloads("f32"):
        name = w.name.split("_")[1]
        st, h = g.gett_log_plan(g.GETT_FLOAT32, w.modes_C, w.shape("C"), None, w.modes_A,
                                w.shape("A"), None, w.modes_B, w.shape("B"), None)
        if h:
            g.gett_log_destroy(h)
        assert (st == 0) == paper[name], name
        assert st in (0, g.GETT_ERROR_NOT_SUPPORTED)


@pytest.mark.parametrize("dtype", ["f32", "f64"])
def test_every_contraction_plans(dtype):
    code = g.GETT_FLOAT32 if dtype == "f32" else g.GETT_FLOAT64
    for w in appendix_workloads(dtype):
        args = (w.modes_C, w.shape("C"), None, w.modes_A, w.shape("A"), None, w.modes_B,
                w.shape("B"), None)
        st, h = g.gett_plan(code, *args, 0)
        assert st == 0, w.name
        d = json.loads(g.gett_plan_describe(h))
        g.gett_destroy(h)
        assert d["flops"] == wl.flop_count(w)
        st, h = g.gett_ttgt_plan(code, *args, -1)
        assert st == 0, w.name
        g.gett_ttgt_destroy(h)
