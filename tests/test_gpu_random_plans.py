"""Randomised parity across the plan's choices at once: random contractions
(ranks up to 6, some with long contracted sets, ragged extents), random
layouts (dense, gapped, permuted), random alpha / beta, and a random forced
choice of tile, kernel kind (macro-kernel, streaming kernel, K slices with a
random count) and flags (no operand exchange, element-wise accesses, no
index split, deterministic) -- every combination against the oracle, and
integer-valued inputs exactly."""
import numpy as np
import pytest

import paper_1607_00145_amd as g
import workloads as wl
from gpu_util import split
from test_gpu_parity import TILES, check_case

pytestmark = pytest.mark.gpu

FLAGS = [0, g.GETT_FLAG_NO_SWAP, g.GETT_FLAG_SCALAR, g.GETT_FLAG_NO_SPLIT,
         g.GETT_FLAG_DETERMINISTIC, g.GETT_FLAG_NO_SWAP | g.GETT_FLAG_NO_SPLIT]


def draw(seed):
    rng = np.random.default_rng(90_000 + seed)
    deep = seed % 3 == 0
    mc, ma, mb, ext = wl.random_problem(rng, max_rank=6, max_ext=9,
                                        allow_empty_sets=(seed % 11 == 10))
    if deep:   # stretch the contracted set so that K boxes (and slices) repeat
        for x in split(ma):
            if x not in split(mc):
                ext[x] = int(rng.integers(20, 70))
                break
    dtype = np.float32 if seed % 2 == 0 else np.float64
    tile = int(rng.integers(0, TILES[dtype]))
    kind = int(rng.integers(0, 3))
    slices = int(rng.integers(2, 17)) if kind == 2 else None
    flags = FLAGS[int(rng.integers(0, len(FLAGS)))]
    kinds = tuple(rng.choice(["dense", "gapped", "permuted"]) for _ in range(3))
    alpha = float(rng.choice([1.0, -0.5, 2.0, 0.0 if seed % 13 == 0 else 1.5]))
    beta = float(rng.choice([0.0, 1.0, -1.5]))
    dist = "int" if seed % 4 == 1 else "uniform"
    return rng, (mc, ma, mb), ext, dtype, tile, kind, slices, flags, kinds, alpha, beta, dist


@pytest.mark.parametrize("seed", range(96))
def test_random_plan_choices(gpu, monkeypatch, seed):
    rng, modes, ext, dtype, tile, kind, slices, flags, kinds, alpha, beta, dist = draw(seed)
    monkeypatch.setenv("GETT_FORCE_TILE", str(tile))
    monkeypatch.setenv("GETT_FORCE_KIND", str(min(kind, 1)))
    if slices:
        monkeypatch.setenv("GETT_FORCE_KSLICES", str(slices))
    shp = lambda m: [ext[x] for x in split(m)]
    got, ref = check_case(gpu, rng, modes, (shp(modes[0]), shp(modes[1]), shp(modes[2])), dtype,
                          alpha, beta, kinds=kinds, flags=flags, dist=dist)
    if dist == "int":
        np.testing.assert_array_equal(got.astype(np.float64), ref.out64)
