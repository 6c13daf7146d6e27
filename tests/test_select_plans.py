"""Method selection plans (host only, Sec. 6): which of GETT, TTGT and LoG
are candidates for a contraction -- exactly those whose own planners accept
it, TTGT within the workspace cap -- the starting method, forcing, and
error handling."""
import json

import pytest

import paper_1607_00145_amd as g

CASES = [
    # (modes C, A, B), extents
    (("ab", "ac", "cb"), {"a": 40, "b": 30, "c": 20}),          # a GEMM: all three apply
    (("abc", "ack", "bk"), {"a": 33, "b": 20, "c": 7, "k": 45}),  # TTGT transposes C
    (("abij", "iejf", "faeb"), {x: 6 for x in "abijef"}),
    (("abcijk", "dabi", "cdjk"), {x: 5 for x in "abcdijk"}),
    (("abc", "bda", "dc"), {"a": 9, "b": 8, "c": 7, "d": 6}),   # LoG refused: a and b in I_m
]


def plans(modes, ext, cap=-1, dtype=g.GETT_FLOAT64):
    shp = lambda m: [ext[x] for x in m]
    args = (dtype, modes[0], shp(modes[0]), None, modes[1], shp(modes[1]), None, modes[2],
            shp(modes[2]), None)
    st, s = g.gett_select_plan(*args, 0, cap)
    assert st == 0
    st_t, t = g.gett_ttgt_plan(*args, cap)
    st_l, l = g.gett_log_plan(*args)
    ws = g.gett_ttgt_workspace_size(t)[1] if st_t == 0 else 0
    if t:
        g.gett_ttgt_destroy(t)
    if l:
        g.gett_log_destroy(l)
    return s, st_t == 0, st_l == 0, ws


@pytest.mark.parametrize("case", range(len(CASES)))
def test_candidates_follow_the_planners(case):
    modes, ext = CASES[case]
    s, has_t, has_l, ws = plans(modes, ext)
    try:
        d = json.loads(g.gett_select_describe(s))
        assert d["method"] == "gett" and not d["timed"]
        assert d["available"] == {"gett": True, "ttgt": has_t, "log": has_l}
        assert d["workspace_bytes"] == ws == g.gett_select_workspace_size(s)[1]
        assert d["ms"] == {"gett": None, "ttgt": None, "log": None}
        assert g.gett_select_method(s) == (0, g.GETT_METHOD_GETT)
        for m, ok in ((g.GETT_METHOD_TTGT, has_t), (g.GETT_METHOD_LOG, has_l),
                      (g.GETT_METHOD_GETT, True)):
            assert g.gett_select_force(s, m) == (0 if ok else g.GETT_ERROR_NOT_SUPPORTED)
            if ok:
                assert g.gett_select_method(s) == (0, m)
        assert json.loads(g.gett_select_describe(s))["method"] == "gett"
        for bad in (3, 7, -1, -(1 << 31), (1 << 31) - 1):
            assert g.gett_select_force(s, bad) == g.GETT_ERROR_INVALID_VALUE
    finally:
        g.gett_select_destroy(s)


def test_workspace_cap_removes_ttgt():
    modes, ext = CASES[1]
    s, has_t, _, ws = plans(modes, ext)
    g.gett_select_destroy(s)
    assert has_t and ws > 0
    s, has_t, _, _ = plans(modes, ext, cap=ws - 1)
    try:
        assert not has_t
        d = json.loads(g.gett_select_describe(s))
        assert not d["available"]["ttgt"] and d["workspace_bytes"] == 0
        assert g.gett_select_force(s, g.GETT_METHOD_TTGT) == g.GETT_ERROR_NOT_SUPPORTED
    finally:
        g.gett_select_destroy(s)


def test_errors():
    st, s = g.gett_select_plan(g.GETT_FLOAT32, "ab", [3, 4], None, "ac", [3, 5], None, "cd",
                               [5, 4], None)
    assert st == g.GETT_ERROR_INVALID_INDICES and s is None
    assert g.gett_select_destroy(None) == 0
    assert g.gett_select_describe(None) == ""
    assert g.gett_select_method(None)[0] == g.GETT_ERROR_INVALID_VALUE
    assert g.gett_select_workspace_size(None)[0] == g.GETT_ERROR_INVALID_VALUE
    assert g.gett_select_force(None, 0) == g.GETT_ERROR_INVALID_VALUE
    assert g.gett_select_contract(None, 1.0, 0, 0, 0.0, 0, 0, 0) == g.GETT_ERROR_INVALID_VALUE
    modes, ext = CASES[0]
    s, _, _, _ = plans(modes, ext)
    try:
        assert g.gett_select_tune(s, -1, 0, 0, 0, 0, 0) == g.GETT_ERROR_INVALID_VALUE
    finally:
        g.gett_select_destroy(s)
