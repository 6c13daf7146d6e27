"""The whole-C comparison used by the full-size GPU parity tests, checked on
the CPU: chunk boundaries, a wrong element and an unwritten (NaN) element."""
import numpy as np
import pytest

import oracle
import workloads as wl
from gpu_util import TOL, compare_whole


@pytest.mark.parametrize("number,chunk", [(2, 1000), (3, 100), (4, 500)])
def test_compare_whole_on_host_tensor(number, chunk):
    import torch
    w = wl.scaled(wl.WORKLOADS[number - 1],
                  {2: {"a": 9, "b": 7, "c": 5, "d": 6, "e": 4},
                   3: {"a": 5, "b": 4, "i": 6, "j": 3, "e": 4, "f": 5},
                   4: {"a": 3, "b": 4, "c": 5, "d": 6, "i": 2, "j": 3, "k": 4}}[number])
    A, B, Cin = wl.make_inputs(w)
    ref = oracle.contract(w.modes_C, w.modes_A, w.modes_B, A, B, w.alpha, w.beta, Cin,
                          shape_C=w.shape("C"))
    flat = ref.out64.reshape(-1, order="F").astype(w.np_dtype)   # rounded like a GPU result
    t = torch.from_numpy(flat.copy())
    assert compare_whole(t, w, A, B, Cin, chunk=chunk) <= TOL[w.np_dtype]
    bad = t.clone()
    bad[len(flat) - 1] += 0.5                                   # last element, last chunk
    assert compare_whole(bad, w, A, B, Cin, chunk=chunk) > TOL[w.np_dtype]
    bad = t.clone()
    bad[chunk] = float("nan")                                   # first element of a chunk
    assert compare_whole(bad, w, A, B, Cin, chunk=chunk) == float("inf")
