"""GPU parity over the Fig. 11 sweep (Sec. 7.3): both contractions, both
precisions, every S_Ik from 8 to 1024 at full size (S_Im = S_In = 1152),
in the plan the benchmark times.  The oracle checks every element of C;
C starts as NaN, so every element must also have been written."""
import numpy as np
import pytest

import paper_1607_00145_amd as g
import workloads as wl
from gpu_util import TOL, compare_whole

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("k", wl.FIG11_K)
@pytest.mark.parametrize("dtype", ["f32", "f64"])
@pytest.mark.parametrize("variant", ["a", "b"])
def test_fig11_point(gpu, variant, dtype, k):
    import torch
    w = wl.fig11(variant, k, dtype)
    A, B, _ = wl.make_inputs(w)
    flat = lambda t: torch.from_numpy(np.asfortranarray(t).reshape(-1, order="F")).to(gpu)
    tA, tB = flat(A), flat(B)
    nC = w.numel("C")
    tC = torch.full((nC,), float("nan"), dtype=tA.dtype, device=gpu)
    dt = g.GETT_FLOAT32 if dtype == "f32" else g.GETT_FLOAT64
    st, h = g.gett_plan(dt, w.modes_C, w.shape("C"), None, w.modes_A, w.shape("A"), None,
                        w.modes_B, w.shape("B"), None, 0)
    assert st == 0
    try:
        st = g.gett_contract(h, w.alpha, tA.data_ptr(), tB.data_ptr(), w.beta, tC.data_ptr(),
                             torch.cuda.current_stream().cuda_stream)
        assert st == 0
        torch.cuda.synchronize()
    finally:
        g.gett_destroy(h)
    assert bool(torch.isfinite(tC).all()), "some element of C was not written"
    err = compare_whole(tC, w, A, B, None)
    assert err <= TOL[w.np_dtype], f"{w.name}: rel err {err:.3e}"
