"""Helpers shared by the GPU tests: strided operands built on host buffers
that the oracle and the GPU library both see, and the parity check."""
from __future__ import annotations

import numpy as np

import oracle
import paper_1607_00145_amd as g

TOL = {np.float32: 1e-4, np.float64: 1e-12}   # max |diff| / (|alpha| sum|a||b| + |beta||c|)


def split(modes):
    return [m for m in modes.split(",") if m] if "," in modes else list(modes)


class Operand:
    """A tensor stored in a flat host buffer with arbitrary positive strides."""

    def __init__(self, flat: np.ndarray, shape, strides, offset: int = 0):
        self.flat, self.shape, self.strides, self.offset = flat, list(shape), list(strides), offset

    @property
    def view(self) -> np.ndarray:
        it = self.flat.itemsize
        return np.lib.stride_tricks.as_strided(self.flat[self.offset:], self.shape,
                                               [s * it for s in self.strides])

    def device(self, dev):
        import torch
        buf = torch.from_numpy(self.flat).to(dev)
        return buf, torch.as_strided(buf, self.shape, self.strides, self.offset)


def layout(rng, shape, kind: str):
    """Strides for a layout: 'dense' (first index stride-one), 'gapped' (each
    index padded), 'permuted' (dense in a random storage order)."""
    n = len(shape)
    if kind == "dense" or n == 0:
        order = list(range(n))
        pad = [0] * n
    elif kind == "gapped":
        order = list(range(n))
        pad = [int(rng.integers(0, 3)) for _ in range(n)]
    elif kind == "permuted":
        order = list(rng.permutation(n))
        pad = [0] * n
    else:
        raise ValueError(kind)
    strides = [0] * n
    acc = 1
    for i in order:
        strides[i] = acc
        acc *= max(shape[i], 1) + pad[i]
    return strides, acc


def make_operand(rng, shape, dtype, kind="dense", dist="uniform", offset=0, guard=4):
    """Values everywhere in the buffer (gaps and a guard band included)."""
    strides, span = layout(rng, shape, kind)
    size = offset + span + guard
    if dist == "int":
        flat = rng.integers(-4, 5, size=size).astype(dtype)
    else:
        flat = rng.uniform(-1, 1, size=size).astype(dtype)
    return Operand(flat, shape, strides, offset)


def run_gpu(dev, modes, ops, alpha, beta, flags=0, c_init=None):
    """Contract on the GPU through the C interface.  ops = (C, A, B) Operands.
    Returns the whole C buffer after the call (numpy)."""
    import torch
    mc, ma, mb = modes
    C, A, B = ops
    dt = g.GETT_FLOAT32 if C.flat.dtype == np.float32 else g.GETT_FLOAT64
    st, h = g.gett_plan(dt, mc, C.shape, C.strides, ma, A.shape, A.strides, mb, B.shape,
                        B.strides, flags)
    assert st == 0, g.gett_status_string(st)
    try:
        bufC, _ = C.device(dev)
        bufA, _ = A.device(dev)
        bufB, _ = B.device(dev)
        it = C.flat.itemsize
        stream = torch.cuda.current_stream().cuda_stream
        st = g.gett_contract(h, alpha, bufA.data_ptr() + A.offset * it,
                             bufB.data_ptr() + B.offset * it, beta,
                             bufC.data_ptr() + C.offset * it, stream)
        assert st == 0, g.gett_status_string(st)
        torch.cuda.synchronize()
        return bufC.cpu().numpy(), h
    finally:
        g.gett_destroy(h)


def reference(modes, ops, alpha, beta):
    mc, ma, mb = modes
    C, A, B = ops
    return oracle.contract(mc, ma, mb, A.view, B.view, alpha, beta,
                           C.view if beta != 0 else None, shape_C=C.shape)


def result_view(flat, C: Operand):
    return np.lib.stride_tricks.as_strided(flat[C.offset:], C.shape,
                                           [s * flat.itemsize for s in C.strides])


def touched_mask(C: Operand):
    """Boolean mask over C's flat buffer: True where an element of C lives."""
    m = np.zeros(C.flat.size, dtype=bool)
    idx = np.zeros(C.shape, dtype=np.int64) if C.shape else np.zeros((), dtype=np.int64)
    for ax, s in enumerate(C.strides):
        sh = [1] * len(C.shape)
        sh[ax] = C.shape[ax]
        idx = idx + (np.arange(C.shape[ax]) * s).reshape(sh)
    m[C.offset + idx.reshape(-1)] = True
    return m


def compare_whole(tC, w, A, B, Cin, chunk: int = 1 << 24) -> float:
    """Every element of a dense column-major C on the device against the
    oracle (all host threads), in chunks of `chunk` elements so the host
    holds at most a chunk of out64 / den64 at a time.  Returns the largest
    relative error; raises on a non-finite or mismatched element."""
    nC = w.numel("C")
    worst = 0.0
    for lo in range(0, nC, chunk):
        hi = min(nC, lo + chunk)
        got = tC[lo:hi].cpu().numpy()
        ref = oracle.contract(w.modes_C, w.modes_A, w.modes_B, A, B, w.alpha, w.beta, Cin,
                              shape_C=w.shape("C"), points=np.arange(lo, hi, dtype=np.int64))
        worst = max(worst, oracle.rel_error(got, ref))
    return worst
