"""Seeded synthetic workloads for the GETT contraction.

This module only describes problems and draws their inputs.  It holds none of
the contraction's arithmetic: both the GPU library's tests and the oracle take
their inputs from here, and nothing here depends on either of them.

Named workloads (all tensors column-major: the first mode is stride-one, the
paper's Fortran layout of Sec. 2.2).  Each stands in for one family of the
paper's 48-contraction benchmark (Sec. 7.1, Appendix A):

  tm3x2_fp32   C[a,b,c] = A[a,k,c] * B[k,b], all extents 32 -- tensor-matrix
               family, same structure as abc-adc-db.
  bw4x3_fp32   C[a,b,c,d] = A[a,e,b] * B[e,d,c], a..d = 112, e = 16,
               alpha 1.5, beta 1 -- small contracted extent, bandwidth bound.
  cc4x4_fp64   C[a,b,i,j] = A[i,e,j,f] * B[f,a,e,b], all 48, alpha 1, beta 1,
               A,B ~ N(0,1), C_in ~ U[-1,1] -- coupled-cluster 4D x 4D family.
  ccsdt6_fp64  C[a,b,c,i,j,k] = A[d,a,b,i] * B[c,d,j,k], all 24 -- CCSD(T)
               6D-output family with one small contracted index.
  gemm4_fp32   C[m1,n1,m2,n2] = A[m1,k1,m2,k2] * B[k2,n1,k1,n2], all 64 --
               4D x 4D shaped like a 4096^3 GEMM, same structure as
               abcd-aecf-fbed.

Draw order (one numpy PCG64 stream per workload, seed 160700145 + number):
A, then B, then C_in when beta != 0, each as a flat fp64 array in storage
order, then cast to the working type.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, List

import numpy as np

SEED_BASE = 160700145


@dataclass(frozen=True)
class Workload:
    number: int
    name: str
    dtype: str                 # "f32" | "f64"
    modes_C: str               # comma separated mode names
    modes_A: str
    modes_B: str
    extents: Dict[str, int] = field(hash=False)
    alpha: float = 1.0
    beta: float = 0.0
    dist_AB: str = "uniform"   # "uniform" U[-1,1] | "normal" N(0,1)
    dist_C: str = "uniform"

    @property
    def np_dtype(self):
        return np.float32 if self.dtype == "f32" else np.float64

    def modes(self, which: str) -> List[str]:
        s = getattr(self, "modes_" + which)
        return [m for m in s.split(",") if m] if "," in s else list(s)

    def shape(self, which: str) -> List[int]:
        return [self.extents[m] for m in self.modes(which)]

    def numel(self, which: str) -> int:
        return int(np.prod(self.shape(which)))

    @property
    def seed(self) -> int:
        return SEED_BASE + self.number

    def expression(self) -> str:
        return (f"C[{self.modes_C}] = A[{self.modes_A}] * B[{self.modes_B}]")


WORKLOADS: List[Workload] = [
    Workload(1, "tm3x2_fp32", "f32", "a,b,c", "a,k,c", "k,b",
             {m: 32 for m in "abck"}),
    Workload(2, "bw4x3_fp32", "f32", "a,b,c,d", "a,e,b", "e,d,c",
             {"a": 112, "b": 112, "c": 112, "d": 112, "e": 16}, alpha=1.5, beta=1.0),
    Workload(3, "cc4x4_fp64", "f64", "a,b,i,j", "i,e,j,f", "f,a,e,b",
             {m: 48 for m in "abijef"}, alpha=1.0, beta=1.0, dist_AB="normal"),
    Workload(4, "ccsdt6_fp64", "f64", "a,b,c,i,j,k", "d,a,b,i", "c,d,j,k",
             {m: 24 for m in "abcdijk"}),
    Workload(5, "gemm4_fp32", "f32", "m1,n1,m2,n2", "m1,k1,m2,k2", "k2,n1,k1,n2",
             {m: 64 for m in ["m1", "m2", "n1", "n2", "k1", "k2"]}),
]
BY_NAME = {w.name: w for w in WORKLOADS}

# Sec. 7.3, Fig. 11: two contractions with S_Im = S_In = 1152 and S_Ik swept
# from 8 to 1024.  The split of 1152 into two indices is not given; 32 x 36 is
# used for both i1 x i2 and j1 x j2.
FIG11_K = (8, 16, 32, 64, 128, 256, 512, 1024)
FIG11_VARIANTS = {
    # i1 j i2 - i1 k i2 - j k
    "a": ("i1,j,i2", "i1,k,i2", "j,k", {"i1": 32, "i2": 36, "j": 1152}),
    # i1 j1 i2 j2 - i1 k i2 - j1 k j2
    "b": ("i1,j1,i2,j2", "i1,k,i2", "j1,k,j2", {"i1": 32, "i2": 36, "j1": 32, "j2": 36}),
}


def fig11(variant: str, s_ik: int, dtype: str = "f32") -> Workload:
    """One point of the Fig. 11 sweep (alpha 1, beta 0, U[-1,1] inputs)."""
    mc, ma, mb, ext = FIG11_VARIANTS[variant]
    ext = dict(ext, k=int(s_ik))
    number = 100 + 20 * (ord(variant) - ord("a")) + FIG11_K.index(s_ik) if s_ik in FIG11_K \
        else 1000 + int(s_ik)
    if dtype == "f64":
        number += 10
    return Workload(number, f"fig11{variant}_k{s_ik}_{'fp32' if dtype == 'f32' else 'fp64'}",
                    dtype, mc, ma, mb, ext)


def _draw(rng: np.random.Generator, n: int, dist: str) -> np.ndarray:
    if dist == "uniform":
        return rng.uniform(-1.0, 1.0, size=n)
    if dist == "normal":
        return rng.standard_normal(size=n)
    if dist == "int4":   # integers in [-4, 4]: exact in any summation order
        return rng.integers(-4, 5, size=n).astype(np.float64)
    raise ValueError(dist)


def make_inputs(w: Workload, dist_override: str | None = None):
    """Return (A, B, C_in) as Fortran-ordered numpy arrays of the working type.

    C_in is None when beta == 0 (C is then an output only)."""
    rng = np.random.Generator(np.random.PCG64(w.seed))
    dt = w.np_dtype
    dAB = dist_override or w.dist_AB
    A = _draw(rng, w.numel("A"), dAB).astype(dt).reshape(w.shape("A"), order="F")
    B = _draw(rng, w.numel("B"), dAB).astype(dt).reshape(w.shape("B"), order="F")
    C = None
    if w.beta != 0.0:
        C = _draw(rng, w.numel("C"), dist_override or w.dist_C).astype(dt).reshape(
            w.shape("C"), order="F")
    return A, B, C


def scaled(w: Workload, extents: Dict[str, int], name_suffix: str = "_small") -> Workload:
    """The same contraction structure with other extents (for parity tests)."""
    ext = dict(w.extents)
    ext.update(extents)
    return Workload(w.number, w.name + name_suffix, w.dtype, w.modes_C, w.modes_A,
                    w.modes_B, ext, w.alpha, w.beta, w.dist_AB, w.dist_C)


def flop_count(w: Workload) -> int:
    """2 * S_Im * S_In * S_Ik -- every index is counted once: C's modes and
    the contracted ones (the modes of A that are not in C)."""
    mc = set(w.modes("C"))
    total = 1
    for m in w.modes("C"):
        total *= w.extents[m]
    for m in w.modes("A"):
        if m not in mc:
            total *= w.extents[m]
    return 2 * total


def algorithmic_bytes(w: Workload) -> int:
    """|A| + |B| + |C| * (1 + [beta != 0]) in bytes: every operand element is
    read once and C written once (read too when beta != 0)."""
    item = 4 if w.dtype == "f32" else 8
    c = w.numel("C") * (2 if w.beta != 0 else 1)
    return item * (w.numel("A") + w.numel("B") + c)


def random_problem(rng: np.random.Generator, max_rank: int = 6, max_ext: int = 5,
                   allow_empty_sets: bool = False):
    """A random contraction pattern: (modes_C, modes_A, modes_B, extents).

    Indices are split into I_m, I_n, I_k (each non-empty unless
    allow_empty_sets), then each tensor's modes are shuffled independently."""
    names = [chr(ord("a") + i) for i in range(3 * max_rank)]
    rng.shuffle(names)
    lo = 0 if allow_empty_sets else 1
    while True:
        nm, nn, nk = (int(rng.integers(lo, 4)) for _ in range(3))
        if max(nm + nk, nn + nk, nm + nn) <= max_rank and nm + nn + nk > 0:
            break
    Im, In, Ik = names[:nm], names[nm:nm + nn], names[nm + nn:nm + nn + nk]
    ext = {n: int(rng.integers(1, max_ext + 1)) for n in Im + In + Ik}
    mc = list(Im + In); rng.shuffle(mc)
    ma = list(Im + Ik); rng.shuffle(ma)
    mb = list(In + Ik); rng.shuffle(mb)
    return ",".join(mc), ",".join(ma), ",".join(mb), ext


def rank16_problem(variant: str = "8x8x8"):
    """Contractions whose tensors have 16 modes and whose index sets cannot
    merge (no two indices of a set are neighbours in memory in every tensor
    holding them), so the plan keeps every index:
      "8x8x8"  I_m, I_n, I_k of 8 indices each; C interleaves m and n, A
               interleaves m and k, B holds k in reverse order between the n;
      "15x1x1" C of 16 modes, 15 of them in I_m (A then has 16 modes).
    Returns (modes_C, modes_A, modes_B, extents); a few extents are 3, the
    rest 2."""
    if variant == "8x8x8":
        m = [f"m{i}" for i in range(8)]
        n = [f"n{i}" for i in range(8)]
        k = [f"k{i}" for i in range(8)]
        mc = [x for pair in zip(m, n) for x in pair]
        ma = [x for pair in zip(m, k) for x in pair]
        mb = [x for pair in zip(list(reversed(k)), n) for x in pair]
        ext = {x: 2 for x in m + n + k}
        ext.update({"m0": 3, "n3": 3, "k2": 3})
    elif variant == "15x1x1":
        m = [f"m{i}" for i in range(15)]
        mc = m[:7] + ["n"] + m[7:]
        ma = ["k"] + list(reversed(m))
        mb = ["n", "k"]
        ext = {x: 2 for x in m}
        ext.update({"n": 5, "k": 7, "m4": 3})
    else:
        raise ValueError(variant)
    return ",".join(mc), ",".join(ma), ",".join(mb), ext
