"""GPU parity over the benchmark of Appendix A (48 contractions, Tables III
and IV): GETT, TTGT and LoG (where the paper applies it) against the oracle
at reduced extents the oracle checks in full (every extent capped, so tiles
are ragged), and GETT at the paper's full extents on one contraction of each
rank pattern, 1024 sampled elements, C pre-filled with NaN."""
import math

import numpy as np
import pytest

import oracle
import paper_1607_00145_amd as g
import workloads as wl
from gpu_util import TOL
from test_gpu_log import check_log
from test_gpu_parity import check_case
from test_gpu_ttgt import check_ttgt
from workloads.appendix_a import TABLE, appendix_workloads

pytestmark = pytest.mark.gpu
NAMES = [name for name, _, _, _ in TABLE]


def reduced(w):
    """Caps every extent so that no tensor exceeds 120k elements."""
    for cap in (37, 29, 23, 19, 13, 11, 7, 5, 3):
        ext = {k: min(v, cap) for k, v in w.extents.items()}
        size = lambda t: math.prod(ext[m] for m in w.modes(t))
        if max(size("C"), size("A"), size("B")) <= 120_000:
            return ext
    return ext


@pytest.mark.parametrize("dtype", ["f32", "f64"])
@pytest.mark.parametrize("i", range(48), ids=NAMES)
def test_appendix_reduced(gpu, i, dtype):
    w = appendix_workloads(dtype)[i]
    ext = reduced(w)
    shp = lambda t: [ext[m] for m in w.modes(t)]
    modes = (w.modes_C, w.modes_A, w.modes_B)
    shapes = (shp("C"), shp("A"), shp("B"))
    npdt = np.float32 if dtype == "f32" else np.float64
    rng = np.random.default_rng(w.seed)
    check_case(gpu, rng, modes, shapes, npdt, 1.5, 0.5)
    d = check_ttgt(gpu, rng, modes, shapes, npdt, 1.0, 0.0)
    assert d is not None
    d = check_log(gpu, rng, modes, shapes, npdt, -1.0, 1.0)
    assert (d is not None) == TABLE[i][3]


FAMILIES = [0, 2, 5, 8, 11, 12, 15, 18, 19, 30]


@pytest.mark.parametrize("i", FAMILIES, ids=[NAMES[i] for i in FAMILIES])
def test_appendix_full_size_sampled(gpu, i):
    import torch
    w = appendix_workloads("f32")[i]
    A, B, _ = wl.make_inputs(w)
    flat = lambda t: torch.from_numpy(np.asfortranarray(t).reshape(-1, order="F")).to(gpu)
    tA, tB = flat(A), flat(B)
    nC = w.numel("C")
    tC = torch.full((nC,), float("nan"), dtype=tA.dtype, device=gpu)
    st, h = g.gett_plan(g.GETT_FLOAT32, w.modes_C, w.shape("C"), None, w.modes_A, w.shape("A"),
                        None, w.modes_B, w.shape("B"), None, 0)
    assert st == 0
    try:
        st = g.gett_contract(h, 1.0, tA.data_ptr(), tB.data_ptr(), 0.0, tC.data_ptr(),
                             torch.cuda.current_stream().cuda_stream)
        assert st == 0
        torch.cuda.synchronize()
    finally:
        g.gett_destroy(h)
    assert bool(torch.isfinite(tC).all())
    rng = np.random.default_rng(w.seed + 1)
    pts = np.concatenate([rng.integers(0, nC, 1020), [0, 1, nC - 2, nC - 1]])
    got = tC[torch.from_numpy(pts).to(gpu)].cpu().numpy()
    ref = oracle.contract(w.modes_C, w.modes_A, w.modes_B, A, B, 1.0, 0.0, None,
                          shape_C=w.shape("C"), points=pts)
    assert oracle.rel_error(got, ref) <= TOL[np.float32]
