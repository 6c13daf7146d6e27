"""GPU parity of the split index orders (Sec. 3.2.1, Fig. 5: the sub-tensors
keep the stride-one index of every tensor; Examples 1-2: one index read as
two).  Column split: C's stride-one index and the column operand's
stride-one index are different free indices.  K split: A's and B's
stride-one indices are different contracted indices.  Every tile shape and
kernel kind, ragged tails on every index, against the oracle."""
import json

import numpy as np
import pytest

import paper_1607_00145_amd as g
from gpu_util import split
from test_gpu_parity import check_case

pytestmark = pytest.mark.gpu
DTYPES = [np.float32, np.float64]
TILES = {np.float32: 7, np.float64: 15}

# (modes C, A, B), extents: the index patterns of Appendix A's bandwidth-bound
# rows 1, 3, 7 and 31 and compute-bound rows 28 and 30 at reduced extents
COLUMN = {
    "abc-bda-dc": (("a,b,c", "b,d,a", "d,c"), {"a": 48, "b": 20, "c": 7, "d": 37}),
    "abcd-dbea-ec": (("a,b,c,d", "d,b,e,a", "e,c"), {"a": 24, "b": 5, "c": 9, "d": 12, "e": 19}),
    "abcde-ecbfa-fd": (("a,b,c,d,e", "e,c,b,f,a", "f,d"),
                       {"a": 32, "b": 3, "c": 5, "d": 6, "e": 8, "f": 11}),
    "abcdef-dega-gfbc": (("a,b,c,d,e,f", "d,e,g,a", "g,f,b,c"),
                         {"a": 24, "b": 3, "c": 5, "d": 4, "e": 5, "f": 6, "g": 12}),
}
KSPLIT = {
    "abcd-eafb-fdec": (("a,b,c,d", "e,a,f,b", "f,d,e,c"),
                       {"a": 9, "b": 10, "c": 11, "d": 7, "e": 24, "f": 20}),
    "abcd-eafd-fbec": (("a,b,c,d", "e,a,f,d", "f,b,e,c"),
                       {"a": 13, "b": 6, "c": 10, "d": 5, "e": 16, "f": 12}),
}
CASES = {**COLUMN, **KSPLIT}
# The Y gather the analyser's run-length price model picks at these extents: a
# column split where C keeps long enough write runs, the whole-index order
# where Y is small next to C (abcdef-dega-gfbc: |A| = |C| / 7.5, so shorter C
# runs would cost more than Y's longer read runs save).
EXPECT = {**{n: "row-vector-strided" for n in COLUMN}, **{n: "k-vector-strided" for n in KSPLIT}}
EXPECT["abcdef-dega-gfbc"] = "scalar"
# a block length forced through the tuning hook, for a pattern the model keeps whole
FORCED = {"abcdef-dega-gfbc": 8}


def shapes_of(modes, ext):
    return tuple([ext[x] for x in split(m)] for m in modes)


def describe(modes, ext, dtype, flags=0):
    code = g.GETT_FLOAT32 if dtype == np.float32 else g.GETT_FLOAT64
    sh = shapes_of(modes, ext)
    st, h = g.gett_plan(code, modes[0], sh[0], None, modes[1], sh[1], None, modes[2], sh[2],
                        None, flags)
    assert st == 0
    try:
        return json.loads(g.gett_plan_describe(h))
    finally:
        g.gett_destroy(h)


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("name", list(CASES))
def test_default_plan(gpu, name, dtype):
    modes, ext = CASES[name]
    d = describe(modes, ext, dtype)
    assert d["gather_y"] == EXPECT[name]
    rng = np.random.default_rng(sum(map(ord, name)))
    check_case(gpu, rng, modes, shapes_of(modes, ext), dtype, 1.5, -0.5)


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("name", list(FORCED))
def test_forced_split(gpu, monkeypatch, name, dtype):
    """The split the model declines, forced: the strided gathers still agree
    with the oracle, with and without beta."""
    monkeypatch.setenv("GETT_SPLIT_F", str(FORCED[name]))
    modes, ext = CASES[name]
    assert describe(modes, ext, dtype)["gather_y"] == "row-vector-strided"
    rng = np.random.default_rng(5)
    check_case(gpu, rng, modes, shapes_of(modes, ext), dtype, 1.5, -0.5)
    got, ref = check_case(gpu, rng, modes, shapes_of(modes, ext), dtype, 1.0, 0.0, dist="int")
    np.testing.assert_array_equal(got.astype(np.float64), ref.out64)


@pytest.mark.parametrize("dtype,tile", [(dt, t) for dt in DTYPES for t in range(TILES[dt])])
@pytest.mark.parametrize("kind", [0, 1])
@pytest.mark.parametrize("name", list(CASES))
def test_every_tile_shape(gpu, monkeypatch, name, dtype, tile, kind):
    monkeypatch.setenv("GETT_FORCE_TILE", str(tile))
    monkeypatch.setenv("GETT_FORCE_KIND", str(kind))
    modes, ext = CASES[name]
    rng = np.random.default_rng(40_000 + 10 * tile + kind)
    beta = 0.0 if kind else 0.75
    check_case(gpu, rng, modes, shapes_of(modes, ext), dtype, -1.25, beta)


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("name", list(CASES))
def test_integer_inputs_bit_exact(gpu, name, dtype):
    modes, ext = CASES[name]
    rng = np.random.default_rng(7)
    got, ref = check_case(gpu, rng, modes, shapes_of(modes, ext), dtype, 1.0, 1.0, dist="int")
    np.testing.assert_array_equal(got.astype(np.float64), ref.out64)


@pytest.mark.parametrize("dtype", DTYPES)
@pytest.mark.parametrize("name", list(CASES))
def test_layouts_and_offsets(gpu, name, dtype):
    """Gapped and permuted layouts (the analyser keeps a split only where
    every vector stays 16-byte aligned) and base pointers off the 16-byte
    grid (vectors dropped at call time)."""
    modes, ext = CASES[name]
    rng = np.random.default_rng(11)
    for kinds, offsets in [(("gapped",) * 3, (0, 0, 0)), (("permuted", "dense", "gapped"), (0, 0, 0)),
                           (("dense",) * 3, (1, 2, 3)), (("dense",) * 3, (0, 1, 0))]:
        check_case(gpu, rng, modes, shapes_of(modes, ext), dtype, 0.5, 2.0, kinds=kinds,
                   offsets=offsets)


@pytest.mark.parametrize("dtype", DTYPES)
def test_no_split_flag_same_result(gpu, dtype):
    """The flag keeps the whole-index order; both plans agree with the
    oracle (and, on integer inputs, with each other exactly)."""
    modes, ext = COLUMN["abc-bda-dc"]
    assert describe(modes, ext, dtype, g.GETT_FLAG_NO_SPLIT)["gather_y"] == "scalar"
    rng = np.random.default_rng(3)
    got0, _ = check_case(gpu, rng, modes, shapes_of(modes, ext), dtype, 1.0, 0.0, dist="int")
    rng = np.random.default_rng(3)
    got1, _ = check_case(gpu, rng, modes, shapes_of(modes, ext), dtype, 1.0, 0.0, dist="int",
                         flags=g.GETT_FLAG_NO_SPLIT)
    np.testing.assert_array_equal(got0, got1)
