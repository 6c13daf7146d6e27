"""Host-side tests of the C interface: the library loads, exports every symbol
the header declares, and the analyser's decisions follow the paper.  No GPU
call is made here (gett_plan is host-only; contract calls either return
before any launch or use the launch fault hook)."""
import json
import os
import re
import subprocess
import sys

import pytest

import paper_1607_00145_amd as g
import workloads as wl

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
GOLDEN = os.path.join(ROOT, "tests", "golden")


def declared_functions():
    text = open(os.path.join(ROOT, "include", "gett.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(gett_\w+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    lib = g.load_library()
    names = declared_functions()
    assert names == sorted(["gett_plan", "gett_contract", "gett_contract_noalloc",
                            "gett_plan_tune", "gett_destroy",
                            "gett_status_string", "gett_plan_describe", "gett_transpose",
                            "gett_ttgt_plan", "gett_ttgt_workspace_size", "gett_ttgt_contract",
                            "gett_ttgt_destroy", "gett_ttgt_describe", "gett_log_plan",
                            "gett_log_contract", "gett_log_destroy", "gett_log_describe",
                            "gett_select_plan", "gett_select_workspace_size", "gett_select_tune",
                            "gett_select_force", "gett_select_method", "gett_select_contract",
                            "gett_select_destroy", "gett_select_describe"])
    for n in names:
        assert hasattr(lib, n), n
    out = subprocess.run(["nm", "-D", "--defined-only", g.LIB_PATH], capture_output=True,
                         text=True).stdout
    for n in names:
        assert re.search(rf"\bT {n}\b", out), n


def test_binding_has_the_c_names():
    for n in declared_functions():
        assert callable(getattr(g, n))


def plan(mc, ma, mb, ext, dtype=g.GETT_FLOAT32, strides=(None, None, None), flags=0):
    sp = lambda m: [x for x in m.split(",") if x] if "," in m else list(m)
    shp = lambda m: [ext[x] for x in sp(m)]
    st, h = g.gett_plan(dtype, mc, shp(mc), strides[0], ma, shp(ma), strides[1], mb, shp(mb),
                        strides[2], flags)
    return st, h


def describe(*a, **k):
    st, h = plan(*a, **k)
    assert st == 0, g.gett_status_string(st)
    d = json.loads(g.gett_plan_describe(h))
    g.gett_destroy(h)
    return d


def test_paper_index_sets():
    """The analyser's I_m / I_n / I_k for every example the paper gives."""
    cases = json.load(open(os.path.join(GOLDEN, "index_sets.json")))["cases"]
    for cs in cases:
        sp = lambda m: [x for x in m.split(",") if x] if "," in m else list(m)
        names = set(sp(cs["C"])) | set(sp(cs["A"])) | set(sp(cs["B"]))
        ext = {n: 3 + i for i, n in enumerate(sorted(names))}   # distinct extents: no merging
        # strided layouts with gaps so that nothing merges either
        strides = []
        for m in (cs["C"], cs["A"], cs["B"]):
            s, acc = [], 1
            for n in sp(m):
                s.append(acc)
                acc *= ext[n] + 1
            strides.append(s)
        d = describe(cs["C"], cs["A"], cs["B"], ext, strides=tuple(strides))
        got = lambda key: sorted(x["name"] for x in d[key])
        assert got("I_m") == sorted(cs["I_m"]), cs["cite"]
        assert got("I_n") == sorted(cs["I_n"]), cs["cite"]
        assert got("I_k") == sorted(cs["I_k"]), cs["cite"]


def test_listing8_super_indices():
    """Sec. 5, Listing 8: for C_abcijk = A_ijmc B_mkab (all 24) the indices a,b
    and i,j merge into super-indices of 576 with the listing's strides."""
    gold = json.load(open(os.path.join(GOLDEN, "listing8_log.json")))
    n = gold["contraction"]["extent"]
    d = describe("abcijk", "ijmc", "mkab", {m: n for m in "abcijkm"})
    assert sorted(d["merges"]) == ["(a,b)", "(i,j)"]
    byname = {x["name"]: x for x in d["I_m"] + d["I_n"] + d["I_k"]}
    assert byname["(a,b)"]["extent"] == gold["super_indices"]["ab"]
    assert byname["(i,j)"]["extent"] == gold["super_indices"]["ij"]
    # leading dimensions of the listing's GEMM: B's (a,b) stride, A's m stride, C's (i,j) stride
    assert byname["(a,b)"]["strideB"] == gold["leading_dims"]["lda_on_B"]
    assert byname["m"]["strideA"] == gold["leading_dims"]["ldb_on_A"]
    assert byname["(i,j)"]["strideC"] == gold["leading_dims"]["ldc"]
    # per-loop offsets of the looped indices c and k
    assert byname["c"]["strideA"] == gold["offsets"]["A_per_c"]
    assert byname["c"]["strideC"] == gold["offsets"]["C_per_c"]
    assert byname["k"]["strideB"] == gold["offsets"]["B_per_k"]
    assert byname["k"]["strideC"] == gold["offsets"]["C_per_k"]
    assert d["size_k"] == gold["gemm"]["k"]


def test_listing6_is_not_merged():
    """Sec. 4, Listing 6: a and c are consecutive in A (a,c,k) but not in C
    (a,b,c), so the super-index merge of footnote 18 must not join them."""
    d = describe("abc", "ack", "bk", {m: 8 for m in "abck"})
    assert d["merges"] == []


def test_workload_plans():
    """The decisions for the five workloads (C's stride-one index on the
    column side; merges of the 6D case; vector gathers along stride-one runs)."""
    exp = {
        1: dict(swapped=True, merges=[], gx="k-vector", gy="row-vector"),
        2: dict(swapped=True, merges=[], gx="k-vector", gy="row-vector"),
        3: dict(swapped=False, merges=[], gx="row-vector", gy="k-vector"),
        4: dict(swapped=True, merges=["(a,b)", "(j,k)"], gx="row-vector", gy="k-vector"),
        5: dict(swapped=True, merges=[], gx="k-vector", gy="row-vector"),
    }
    for w in wl.WORKLOADS:
        dt = g.GETT_FLOAT32 if w.dtype == "f32" else g.GETT_FLOAT64
        d = describe(w.modes_C, w.modes_A, w.modes_B, w.extents, dtype=dt)
        e = exp[w.number]
        assert d["swapped"] == e["swapped"], w.name
        assert sorted(d["merges"]) == e["merges"], w.name
        assert d["gather_x"] == e["gx"] and d["gather_y"] == e["gy"], w.name
        vw = 4 if w.dtype == "f32" else 2
        assert d["c_vector"] is (d["tile"]["reads"][1] == vw)
        assert d["flops"] == wl.flop_count(w)
        # C's stride-one index leads the column order
        first_y = d["y_order"][0]
        strides = {x["name"]: x["strideC"] for x in d["I_m"] + d["I_n"]}
        assert strides[first_y] == 1


def test_flags_change_the_plan():
    w = wl.WORKLOADS[4]
    d0 = describe(w.modes_C, w.modes_A, w.modes_B, w.extents)
    d1 = describe(w.modes_C, w.modes_A, w.modes_B, w.extents, flags=g.GETT_FLAG_NO_SWAP)
    d2 = describe(w.modes_C, w.modes_A, w.modes_B, w.extents, flags=g.GETT_FLAG_SCALAR)
    assert d0["swapped"] and not d1["swapped"]
    assert d2["gather_x"] == d2["gather_y"] == "scalar" and d2["c_vector"] is False


def test_kbox_covers_contracted_set():
    """K boxes tile the contracted index space: steps * box >= S_Ik with the
    block split of one index (index reinterpretation, Sec. 3.2.1)."""
    for ext_k in [(7,), (24,), (48, 48), (3, 5, 2), (64, 64), (1,)]:
        names = [f"k{i}" for i in range(len(ext_k))]
        ext = {"m": 9, "n": 10, **dict(zip(names, ext_k))}
        d = describe("m,n", ",".join(["m"] + names), ",".join(names + ["n"]), ext)
        kb = d["kbox"]
        tot = 1
        for e in ext_k:
            tot *= e
        assert kb["steps"] * kb["elements"] >= tot
        assert kb["elements"] <= d["tile"]["kt"]


@pytest.mark.parametrize("mc,ma,mb,code", [
    ("m,n,b", "m,k,b", "k,n,b", 2),     # batch index in all three (fn. 9)
    ("m,n", "m,k", "n", 2),             # k only in A
    ("m,n,z", "m,k", "k,n", 2),         # z only in C
    ("m,n", "m,m,k", "k,n", 2),         # repeated index
    ("m,n", "m,,k", "k,n", 2),          # empty name
])
def test_invalid_indices(mc, ma, mb, code):
    sp = lambda m: [x for x in m.split(",") if x]
    st, h = g.gett_plan(0, mc, [2] * len(sp(mc)), None, ma, [2] * len(sp(ma)), None, mb,
                        [2] * len(sp(mb)), None, 0)
    assert st == code and h is None


def test_invalid_values_and_unsupported():
    st, _ = g.gett_plan(7, "m,n", [2, 2], None, "m,k", [2, 2], None, "k,n", [2, 2], None)
    assert st == 1                                                  # bad dtype
    st, _ = g.gett_plan(0, "m,n", [2, 3], None, "m,k", [2, 2], None, "k,n", [2, 2], None)
    assert st == 2                                                  # extent mismatch
    st, _ = g.gett_plan(0, "m,n", [-1, 2], None, "m,k", [-1, 2], None, "k,n", [2, 2], None)
    assert st == 1                                                  # negative extent
    st, _ = g.gett_plan(0, "m,n", [4, 4], [1, 2], "m,k", [4, 2], None, "k,n", [2, 4], None)
    assert st == 3                                                  # overlapping C
    st, _ = g.gett_plan(0, "m,n", [4, 4], [0, 4], "m,k", [4, 2], None, "k,n", [2, 4], None)
    assert st == 1                                                  # zero stride
    big = 1 << 16
    st, h = g.gett_plan(0, "m,n", [big, big], None, "m,k", [big, 2], None, "k,n", [2, big], None)
    assert st == 0                                                  # C of 2^32 elements
    g.gett_destroy(h)
    st, _ = g.gett_plan(0, "m,n", [1 << 20, 4], [1, 1 << 30], "m,k", [1 << 20, 2], None, "k,n",
                        [2, 4], None)
    assert st == 3                                                  # one tile spans > 2^31
    modes = ",".join(f"i{i}" for i in range(17))
    st, _ = g.gett_plan(0, modes, [1] * 17, None, "k,", [1], None, "k,", [1], None)
    assert st == 3                                                  # rank > GETT_MAX_RANK


def test_contract_host_side_errors():
    st, h = plan("m,n", "m,k", "k,n", {"m": 8, "n": 8, "k": 8})
    assert st == 0
    assert g.gett_contract(None, 1.0, 0x1000, 0x2000, 0.0, 0x3000) == 1   # null plan
    assert g.gett_contract(h, 1.0, 0x1000, 0x2000, 0.0, 0) == 1           # null C
    assert g.gett_contract(h, 1.0, 0, 0x2000, 0.0, 0x3000) == 1           # null A
    assert g.gett_contract(h, 1.0, 0x1001, 0x2000, 0.0, 0x3000) == 1      # misaligned
    assert g.gett_contract(h, 1.0, 0x1000, 0x2000, 0.0, 0x1010) == 1      # C overlaps A
    g.gett_destroy(h)
    assert g.gett_destroy(None) == 0
    assert g.gett_plan_describe(None) == ""
    assert g.gett_status_string(4) == "HIP runtime error"


@pytest.mark.parametrize("value", [2, 7, -1, -(1 << 31), (1 << 31) - 1])
def test_any_int_of_the_enumerations_is_refused_not_undefined(value):
    """The enumerations take the range of a 32-bit int (two range
    enumerators), so an unknown value from a C caller is a value of the type
    and refused; the sanitizer build checks that no load of one is undefined."""
    st, h = g.gett_plan(value, "m,n", [2, 2], None, "m,k", [2, 2], None, "k,n", [2, 2], None)
    assert st == g.GETT_ERROR_INVALID_VALUE and h is None
    E = g.GETT_ERROR_INVALID_VALUE
    assert g.gett_transpose(value, [2, 3], None, [3, 1], 1.0, 0x1000, 0.0, 0x2000) == E


@pytest.mark.parametrize("value", [6, 99, -1, -(1 << 31), (1 << 31) - 1])
def test_unknown_status_has_text(value):
    assert g.gett_status_string(value) == "unknown status"


def test_contract_empty_c_is_a_no_op():
    st, h = plan("m,n", "m,k", "k,n", {"m": 0, "n": 8, "k": 8})
    assert st == 0
    assert json.loads(g.gett_plan_describe(h))["empty_c"] is True
    assert g.gett_contract(h, 1.0, 0x1000, 0x2000, 0.0, 0x3000) == 0
    g.gett_destroy(h)


def test_launch_failure_is_reported():
    """The launch error path, forced from the host (no GPU call happens)."""
    code = (
        "import os, sys; sys.path.insert(0, %r);"
        "import paper_1607_00145_amd as g;"
        "st, h = g.gett_plan(0, 'm,n', [8, 8], None, 'm,k', [8, 8], None, 'k,n', [8, 8], None);"
        "print(g.gett_contract(h, 1.0, 0x10000, 0x20000, 0.0, 0x30000))" % ROOT)
    env = dict(os.environ, GETT_FAULT_INJECT="launch")
    out = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True)
    assert out.stdout.strip() == "4", out.stderr


def test_expression_parser():
    assert g.parse_expression("C[a,b,i,j] = A[i,m,a] * B[m,j,b]") == ("a,b,i,j", "i,m,a", "m,j,b")
    assert g.parse_expression("C[m1] = A[m1,k] * B[k]") == ("m1,", "m1,k", "k,")


def test_candidates_are_ranked_by_the_model():
    """Sec. 3.4: every compiled candidate gets a model estimate; the plan uses
    the cheapest one unless told otherwise."""
    for w in wl.WORKLOADS:
        dt = g.GETT_FLOAT32 if w.dtype == "f32" else g.GETT_FLOAT64
        st, h = plan(w.modes_C, w.modes_A, w.modes_B, w.extents, dtype=dt)
        assert st == 0
        d = json.loads(g.gett_plan_describe(h))
        g.gett_destroy(h)
        cands = d["candidates"]
        assert len(cands) >= 2
        costs = [c["model_us"] for c in cands]
        assert costs == sorted(costs)
        assert all(c > 0 for c in costs)
        assert len({(c["tile"], c["kind"]) for c in cands}) == len(cands)
        assert d["tile"]["chosen_by"] == "model"
        kind = "kslices" if d["kslices"] > 1 else d["kernel"]
        assert (cands[0]["tile"], cands[0]["kind"]) == (d["tile"]["id"], kind)
        assert d["tile"]["model_us"] == costs[0]


def test_forced_candidate_is_reported():
    code = ("import json, paper_1607_00145_amd as g\n"
            "st, h = g.gett_plan(0, 'mn', [300, 200], None, 'mk', [300, 64], None, 'kn', [64, 200], None, 0)\n"
            "d = json.loads(g.gett_plan_describe(h))\n"
            "print(d['tile']['id'], d['tile']['chosen_by'])\n")
    env = dict(os.environ, GETT_FORCE_TILE="0", GETT_FORCE_KIND="0", PYTHONPATH=ROOT)
    out = subprocess.run([sys.executable, "-c", code], env=env, capture_output=True, text=True,
                         cwd=ROOT)
    assert out.returncode == 0, out.stderr
    assert out.stdout.split() == ["0", "forced"]


def test_tune_host_side_errors():
    """gett_plan_tune rejects bad arguments before any HIP call."""
    st, h = plan("mn", "mk", "kn", {"m": 100, "n": 200, "k": 300})
    assert st == 0
    try:
        assert g.gett_plan_tune(None, 4, 256, 1 << 20, 2 << 20) == g.GETT_ERROR_INVALID_VALUE
        assert g.gett_plan_tune(h, 0, 256, 1 << 20, 2 << 20) == g.GETT_ERROR_INVALID_VALUE
        assert g.gett_plan_tune(h, -3, 256, 1 << 20, 2 << 20) == g.GETT_ERROR_INVALID_VALUE
        assert g.gett_plan_tune(h, 4, 0, 1 << 20, 2 << 20) == g.GETT_ERROR_INVALID_VALUE
        assert g.gett_plan_tune(h, 4, 256, 1 << 20, 0) == g.GETT_ERROR_INVALID_VALUE
        assert g.gett_plan_tune(h, 4, 258, 1 << 20, 2 << 20) == g.GETT_ERROR_INVALID_VALUE
        # C overlapping A
        assert g.gett_plan_tune(h, 4, 1 << 20, 4 << 20, (1 << 20) + 64) == \
            g.GETT_ERROR_INVALID_VALUE
        assert json.loads(g.gett_plan_describe(h))["tile"]["chosen_by"] == "model"
    finally:
        g.gett_destroy(h)
    # an empty C: nothing to tune, nothing to check
    st, h = plan("mn", "mk", "kn", {"m": 0, "n": 200, "k": 300})
    assert st == 0
    assert g.gett_plan_tune(h, 4, 0, 0, 0) == g.GETT_SUCCESS
    g.gett_destroy(h)


@pytest.mark.parametrize("variant", ["a", "b"])
def test_fig11_sweep_plans(variant):
    """Sec. 7.3, Fig. 11: S_Im = S_In = 1152 at every S_Ik of the sweep; C's
    stride-one index i1 belongs to A, so the operands are exchanged."""
    for k in wl.FIG11_K:
        w = wl.fig11(variant, k)
        assert wl.flop_count(w) == 2 * 1152 * 1152 * k
        d = describe(w.modes_C, w.modes_A, w.modes_B, w.extents)
        names = lambda key: sorted(x["name"] for x in d[key])
        assert names("I_m") == ["i1", "i2"]
        assert names("I_n") == (["j"] if variant == "a" else ["j1", "j2"])
        assert names("I_k") == ["k"]
        assert d["merges"] == []
        assert d["swapped"] is True
        assert d["size_x"] * d["size_y"] == 1152 * 1152 and d["size_k"] == k


# ------------------------------------------------------------------ TTGT ---

def ttgt_plan(mc, ma, mb, ext, dtype=g.GETT_FLOAT32, strides=(None, None, None), cap=-1):
    shp = lambda m: [ext[x] for x in (m.split(",") if "," in m else list(m)) if x]
    return g.gett_ttgt_plan(dtype, mc, shp(mc), strides[0], ma, shp(ma), strides[1], mb, shp(mb),
                            strides[2], cap)


def ttgt_describe(*a, **k):
    st, h = ttgt_plan(*a, **k)
    assert st == 0, g.gett_status_string(st)
    d = json.loads(g.gett_ttgt_describe(h))
    st, ws = g.gett_ttgt_workspace_size(h)
    assert st == 0 and ws == d["workspace_bytes"]
    g.gett_ttgt_destroy(h)
    return d


def test_ttgt_listing6_example():
    """Sec. 4, Listing 6: for C_abc = A_ack B_bk neither operand needs a
    transposition -- (a,c) is a super-index of A's rows -- and the product
    (a,c) x b is folded into C."""
    ext = {"a": 5, "b": 6, "c": 7, "k": 8}
    d = ttgt_describe("abc", "ack", "bk", ext)
    assert d["transposed"] == ["C"]
    assert d["transposed_elements"] == 5 * 6 * 7
    assert d["order_m"] == "a,c" and d["gemm"]["left"] == "A"
    assert d["gemm"]["op_left"] == "N" and d["gemm"]["op_right"] == "T"
    assert (d["gemm"]["m"], d["gemm"]["n"], d["gemm"]["k"]) == (35, 6, 8)
    assert d["stride_one_changes"] == 0
    assert d["workspace_bytes"] == ((5 * 6 * 7 * 4 + 255) // 256) * 256


def test_ttgt_gemm_shaped_needs_nothing():
    for mc, ma, mb, ops in (("mn", "mk", "kn", ("N", "N")), ("mn", "km", "kn", ("T", "N")),
                            ("mn", "mk", "nk", ("N", "T")), ("nm", "mk", "kn", None)):
        d = ttgt_describe(mc, ma, mb, {"m": 9, "n": 10, "k": 11})
        assert d["transposed"] == [], (mc, ma, mb)
        assert d["workspace_bytes"] == 0
        if ops:
            assert (d["gemm"]["op_left"], d["gemm"]["op_right"]) == ops
        else:   # C = X^T: B is the left operand
            assert d["gemm"]["left"] == "B"


def test_ttgt_plans_of_workloads():
    """The flattening of each workload: the fewest elements transposed.  A
    tensor whose free and contracted indices interleave (A and B of cc4x4, B
    and C of ccsdt6, all three of gemm4) must be transposed whatever the
    arrangement; tm3x2's A (a,k,c) and C (a,b,c) interleave too."""
    exp = {1: ["A", "C"], 2: ["A", "B"], 3: ["A", "B"], 4: ["B", "C"], 5: ["A", "B", "C"]}
    for w in wl.WORKLOADS:
        dt = g.GETT_FLOAT32 if w.dtype == "f32" else g.GETT_FLOAT64
        d = ttgt_describe(w.modes_C, w.modes_A, w.modes_B, w.extents, dtype=dt)
        assert sorted(d["transposed"]) == exp[w.number], (w.name, d)
        na, nb, nc = w.numel("A"), w.numel("B"), w.numel("C")
        size = {"A": na, "B": nb, "C": nc}
        assert d["transposed_elements"] == sum(size[t] for t in d["transposed"])
        m, n, k = d["gemm"]["m"], d["gemm"]["n"], d["gemm"]["k"]
        assert m * n * k * 2 == wl.flop_count(w)


def test_ttgt_workspace_cap():
    ext = {"a": 5, "b": 6, "c": 7, "k": 8}
    st, h = ttgt_plan("abc", "ack", "bk", ext, cap=100)
    assert st == g.GETT_ERROR_NOT_SUPPORTED and h is None
    st, h = ttgt_plan("mn", "mk", "kn", {"m": 9, "n": 10, "k": 11}, cap=0)
    assert st == 0
    g.gett_ttgt_destroy(h)


@pytest.mark.parametrize("mc,ma,mb,code", [("ab", "ak", "kb,", 2), ("ab", "ak", "bk", 0),
                                           ("abk", "ak", "bk", 2), ("ab", "aak", "bk", 2)])
def test_ttgt_plan_validation(mc, ma, mb, code):
    st, h = ttgt_plan(mc, ma, mb, {"a": 3, "b": 4, "k": 5, "kb": 5})
    assert st == code
    if h:
        g.gett_ttgt_destroy(h)


def test_ttgt_contract_host_side_errors():
    st, h = ttgt_plan("abc", "ack", "bk", {"a": 5, "b": 6, "c": 7, "k": 8})
    assert st == 0
    _, ws = g.gett_ttgt_workspace_size(h)
    A, B, C, W = 1 << 20, 2 << 20, 3 << 20, 4 << 20
    try:
        assert g.gett_ttgt_contract(None, 1, A, B, 0, C, W, ws) == g.GETT_ERROR_INVALID_VALUE
        assert g.gett_ttgt_contract(h, 1, A, B, 0, C, 0, ws) == g.GETT_ERROR_INVALID_VALUE
        assert g.gett_ttgt_contract(h, 1, A, B, 0, C, W, ws - 1) == g.GETT_ERROR_INVALID_VALUE
        assert g.gett_ttgt_contract(h, 1, A, B, 0, C, W + 64, ws) == g.GETT_ERROR_INVALID_VALUE
        assert g.gett_ttgt_contract(h, 1, A, B, 0, C, C, ws) == g.GETT_ERROR_INVALID_VALUE
        assert g.gett_ttgt_contract(h, 1, A, B, 0, 0, W, ws) == g.GETT_ERROR_INVALID_VALUE
        assert g.gett_ttgt_contract(h, 1, A, B + 2, 0, C, W, ws) == g.GETT_ERROR_INVALID_VALUE
    finally:
        g.gett_ttgt_destroy(h)
    st, h = ttgt_plan("abc", "ack", "bk", {"a": 0, "b": 6, "c": 7, "k": 8})
    assert st == 0
    assert g.gett_ttgt_contract(h, 1, 0, 0, 0, 0, 0, 0) == g.GETT_SUCCESS   # empty C
    g.gett_ttgt_destroy(h)
    assert g.gett_ttgt_describe(None) == ""
    assert g.gett_ttgt_destroy(None) == g.GETT_SUCCESS


def test_transpose_host_side_errors():
    P, Q = 1 << 20, 2 << 20
    f32 = g.GETT_FLOAT32
    E = g.GETT_ERROR_INVALID_VALUE
    assert g.gett_transpose(7, [2, 3], None, [3, 1], 1, P, 0, Q) == E
    assert g.gett_transpose(f32, [2, -3], None, None, 1, P, 0, Q) == E
    assert g.gett_transpose(f32, [2, 3], [0, 2], None, 1, P, 0, Q) == E
    assert g.gett_transpose(f32, [2, 3], None, [3, 1], 1, P, 0, 0) == E
    assert g.gett_transpose(f32, [2, 3], None, [3, 1], 1, 0, 0, Q) == E
    assert g.gett_transpose(f32, [2, 3], None, [3, 1], 1, P + 2, 0, Q) == E
    assert g.gett_transpose(f32, [2, 3], None, [3, 1], 1, P, 0, P + 8) == E        # overlap
    assert g.gett_transpose(f32, [2] * 17, None, None, 1, P, 0, Q) == g.GETT_ERROR_NOT_SUPPORTED
    assert g.gett_transpose(f32, [2, 2], None, [1, 1], 1, P, 0, Q) == \
        g.GETT_ERROR_NOT_SUPPORTED                                                 # not injective
    assert g.gett_transpose(f32, [1 << 16, 1 << 16], None, None, 1, P, 0, Q) == \
        g.GETT_ERROR_NOT_SUPPORTED                                                 # offset >= 2^31
    assert g.gett_transpose(f32, [2, 0, 3], None, None, 1, P, 0, Q) == g.GETT_SUCCESS   # empty


# ------------------------------------------------------------------- LoG ---

def log_plan(mc, ma, mb, ext, dtype=g.GETT_FLOAT32, strides=(None, None, None)):
    shp = lambda m: [ext[x] for x in (m.split(",") if "," in m else list(m)) if x]
    return g.gett_log_plan(dtype, mc, shp(mc), strides[0], ma, shp(ma), strides[1], mb, shp(mb),
                           strides[2])


def log_describe(*a, **k):
    st, h = log_plan(*a, **k)
    assert st == 0, g.gett_status_string(st)
    d = json.loads(g.gett_log_describe(h))
    g.gett_log_destroy(h)
    return d


def test_log_listing8_plan():
    """Sec. 5, Listing 8: the LoG code printed for C_abcijk = A_ijmc B_mkab
    (all 24) -- operands exchanged, GEMM C_(ab),(ij) = B^T A^T with the
    listing's sizes and leading dimensions, loops over c and k."""
    gold = json.load(open(os.path.join(GOLDEN, "listing8_log.json")))
    c = gold["contraction"]
    d = log_describe(c["C"], c["A"], c["B"], {x: c["extent"] for x in "abcijkm"})
    gm = d["gemm"]
    assert d["swapped"] is True
    assert (gm["m"], gm["n"], gm["k"]) == (gold["gemm"]["m"], gold["gemm"]["n"], gold["gemm"]["k"])
    assert (gm["op_left"], gm["op_right"]) == (gold["gemm"]["transA"], gold["gemm"]["transB"])
    ld = gold["leading_dims"]
    assert (gm["lda"], gm["ldb"], gm["ldc"]) == (ld["lda_on_B"], ld["ldb_on_A"], ld["ldc"])
    assert (gm["m_index"], gm["n_index"], gm["k_index"]) == ("(a,b)", "(i,j)", "m")
    loops = sorted([d["batch"]["index"]] + d["free_loops"] + d["contracted_loops"])
    assert loops == sorted(gold["loops"])
    off = gold["offsets"]
    per = {"k": (off["B_per_k"], off["C_per_k"]), "c": (off["A_per_c"], off["C_per_c"])}
    b = d["batch"]
    assert (b["stride_left"] or b["stride_right"], b["stride_c"]) == per[b["index"]]
    assert d["gemm_calls"] == 24


def test_log_not_applicable():
    """Listing 7: two stride-one indices in one set (a of C and c of A are
    both in I_m) leave no slice with one unit-stride dimension."""
    st, h = log_plan("abc", "cak", "kb", {"a": 4, "b": 5, "c": 6, "k": 7})
    assert st == g.GETT_ERROR_NOT_SUPPORTED and h is None
    st, h = log_plan("ab", "ka", "kb", {"a": 4, "b": 5, "k": 7}, strides=(None, [9, 1], None))
    assert st == 0   # A's stride-one index k is contracted, as B's: same index, allowed
    g.gett_log_destroy(h)


def test_log_gemm_and_swap():
    d = log_describe("mn", "mk", "kn", {"m": 9, "n": 10, "k": 11})
    assert d["batch"] is None and d["free_loops"] == [] and d["gemm_calls"] == 1
    assert (d["gemm"]["op_left"], d["gemm"]["op_right"]) == ("N", "N")
    d = log_describe("nm", "mk", "kn", {"m": 9, "n": 10, "k": 11})
    assert d["swapped"] is True        # C's stride-one index n belongs to B
    assert d["gemm"]["m_index"] == "n"


@pytest.mark.parametrize("variant", ["a", "b"])
def test_log_fig11_slices(variant):
    """Sec. 7.3: for i1 j i2 - i1 k i2 - j k the GEMM's n is S_j = 1152; for
    i1 j1 i2 j2 - i1 k i2 - j1 k j2 it is only S_j1 (smaller GEMMs)."""
    w = wl.fig11(variant, 64)
    d = log_describe(w.modes_C, w.modes_A, w.modes_B, w.extents)
    assert d["gemm"]["m_index"] == "i1" and d["gemm"]["k_index"] == "k"
    if variant == "a":
        assert d["gemm"]["n"] == 1152 and d["batch"]["index"] == "i2" and d["gemm_calls"] == 1
    else:
        assert d["gemm"]["n_index"] == "j1" and d["gemm"]["n"] == 32
        assert d["gemm_calls"] == 36


def test_log_plans_of_workloads():
    for w in wl.WORKLOADS:
        dt = g.GETT_FLOAT32 if w.dtype == "f32" else g.GETT_FLOAT64
        d = log_describe(w.modes_C, w.modes_A, w.modes_B, w.extents, dtype=dt)
        gm = d["gemm"]
        batch = d["batch"]["count"] if d["batch"] else 1
        assert 2 * gm["m"] * gm["n"] * gm["k"] * batch * d["gemm_calls"] == wl.flop_count(w), w.name


def test_log_contract_host_side_errors():
    st, h = log_plan("abc", "akc", "kb", {"a": 5, "b": 6, "c": 7, "k": 8})
    assert st == 0
    try:
        assert g.gett_log_contract(None, 1, 1 << 20, 2 << 20, 0, 3 << 20) == g.GETT_ERROR_INVALID_VALUE
        assert g.gett_log_contract(h, 1, 1 << 20, 2 << 20, 0, 0) == g.GETT_ERROR_INVALID_VALUE
        assert g.gett_log_contract(h, 1, 0, 2 << 20, 0, 3 << 20) == g.GETT_ERROR_INVALID_VALUE
        assert g.gett_log_contract(h, 1, 1 << 20, 2 << 20, 0, (1 << 20) + 4) == \
            g.GETT_ERROR_INVALID_VALUE
    finally:
        g.gett_log_destroy(h)
    assert g.gett_log_describe(None) == "" and g.gett_log_destroy(None) == 0


@pytest.mark.parametrize("variant", ["8x8x8", "15x1x1"])
@pytest.mark.parametrize("dtype", [g.GETT_FLOAT32, g.GETT_FLOAT64])
def test_rank16_plans_keep_every_index(variant, dtype):
    """Tensors of 16 modes (GETT_MAX_RANK; Sec. 2.2 allows any order) plan
    with every index kept: no two indices of a set are memory neighbours in
    all the tensors that hold them."""
    mc, ma, mb, ext = wl.rank16_problem(variant)
    d = describe(mc, ma, mb, ext, dtype=dtype)
    sizes = {"8x8x8": (8, 8, 8), "15x1x1": (15, 1, 1)}[variant]
    assert (len(d["I_m"]), len(d["I_n"]), len(d["I_k"])) == sizes
    assert d["merges"] == []
    assert max(len(d["x_order"]), len(d["y_order"])) == max(sizes[0], sizes[1])


def test_hooks_are_part_of_the_plan(monkeypatch):
    """The tuning hooks in force are listed by the description (sanitised for
    JSON) and change nothing when unset."""
    monkeypatch.delenv("GETT_FORCE_TILE", raising=False)
    st, h = plan("m,n", "m,k", "k,n", {"m": 64, "n": 64, "k": 64})
    d0 = json.loads(g.gett_plan_describe(h))
    g.gett_destroy(h)
    assert d0["hooks"] == ""
    monkeypatch.setenv("GETT_FORCE_TILE", "3")
    monkeypatch.setenv("GETT_SPLIT_F", 'x"y')
    st, h = plan("m,n", "m,k", "k,n", {"m": 64, "n": 64, "k": 64})
    d1 = json.loads(g.gett_plan_describe(h))
    g.gett_destroy(h)
    assert "GETT_FORCE_TILE=3;" in d1["hooks"] and "GETT_SPLIT_F=x?y;" in d1["hooks"]
    assert d1["tile"]["id"] == 3 and d1["tile"]["chosen_by"] == "forced"
