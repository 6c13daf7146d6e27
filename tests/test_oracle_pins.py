"""Pins of the oracle against what the paper and the mathematics fix.

Every check here compares the oracle (``oracle/gett_oracle.c``) with something
that is not the oracle: a literal Python loop, numpy's einsum and matmul, a
GEMM written out by definition (Listing 1), closed forms, the TTGT
decomposition (Sec. 4) and the Loops-over-GEMM code printed in Listing 8.
"""
import itertools
import json
import math
import os

import numpy as np
import pytest

import oracle
import workloads as wl

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


# ---------------------------------------------------------------- helpers ---

def split(modes):
    """Comma-separated names (a trailing comma marks a single name), else one
    character per mode."""
    return [m for m in modes.split(",") if m] if "," in modes else list(modes)


def brute_force(mc, ma, mb, ext, A, B, alpha, beta, C):
    """Eq. 2 as literal Python loops over every index (tiny inputs only)."""
    mc, ma, mb = split(mc), split(ma), split(mb)
    kidx = [m for m in ma if m not in mc]
    out = np.zeros([ext[m] for m in mc]) if mc else np.zeros(())
    for cpos in itertools.product(*[range(ext[m]) for m in mc]):
        val = dict(zip(mc, cpos))
        t = 0.0
        for kpos in itertools.product(*[range(ext[m]) for m in kidx]):
            val.update(zip(kidx, kpos))
            t += float(A[tuple(val[m] for m in ma)]) * float(B[tuple(val[m] for m in mb)])
        r = alpha * t
        if beta != 0:
            r += beta * float(C[cpos])
        out[cpos] = r
    return out


def einsum_ref(mc, ma, mb, A, B, alpha, beta, C):
    mc, ma, mb = split(mc), split(ma), split(mb)
    letters = {}
    for m in mc + ma + mb:
        letters.setdefault(m, chr(ord("a") + len(letters)))
    spec = "".join(letters[m] for m in ma) + "," + "".join(letters[m] for m in mb) + "->" + \
        "".join(letters[m] for m in mc)
    t = np.einsum(spec, A.astype(np.float64), B.astype(np.float64), optimize=False)
    r = alpha * t
    if beta != 0:
        r = r + beta * C.astype(np.float64)
    return r


def rand(rng, shape, dtype=np.float64, kind="uniform"):
    if kind == "int":
        a = rng.integers(-4, 5, size=shape).astype(dtype)
    else:
        a = rng.uniform(-1, 1, size=shape).astype(dtype)
    return np.asfortranarray(a)


def run(mc, ma, mb, ext, A, B, alpha=1.0, beta=0.0, C=None, **kw):
    shape_c = [ext[m] for m in split(mc)]
    return oracle.contract(mc, ma, mb, A, B, alpha, beta, C, shape_C=shape_c, **kw)


# ------------------------------------------------------------ brute force ---

@pytest.mark.parametrize("seed", range(40))
def test_brute_force_random_patterns(seed):
    """Listing 3 / Eq. 2 by literal loops, every mode pattern up to rank 6."""
    rng = np.random.default_rng(1000 + seed)
    mc, ma, mb, ext = wl.random_problem(rng, max_rank=6, max_ext=3,
                                        allow_empty_sets=(seed % 4 == 0))
    sh = lambda m: [ext[x] for x in split(m)]
    A, B, C = rand(rng, sh(ma)), rand(rng, sh(mb)), rand(rng, sh(mc))
    alpha, beta = float(rng.uniform(-2, 2)), float(rng.choice([0.0, 1.0, -0.5]))
    ref = brute_force(mc, ma, mb, ext, A, B, alpha, beta, C)
    got = run(mc, ma, mb, ext, A, B, alpha, beta, C)
    np.testing.assert_allclose(got.out64, ref, rtol=1e-13, atol=1e-13)


@pytest.mark.parametrize("seed", range(30))
@pytest.mark.parametrize("dtype", [np.float32, np.float64])
def test_einsum_random_strided(seed, dtype):
    """numpy.einsum (no path optimisation, fp64) on non-dense, permuted views."""
    rng = np.random.default_rng(2000 + seed)
    mc, ma, mb, ext = wl.random_problem(rng, max_rank=6, max_ext=5)
    sh = lambda m: [ext[x] for x in split(m)]

    def strided(shape):
        # a view with gaps: allocate a larger array and slice every other element
        big = rand(rng, [2 * s for s in shape], dtype)
        return big[tuple(slice(0, 2 * s, 2) for s in shape)]

    A, B, C = strided(sh(ma)), strided(sh(mb)), strided(sh(mc))
    alpha, beta = 1.25, float(rng.choice([0.0, 0.75]))
    ref = einsum_ref(mc, ma, mb, A, B, alpha, beta, C)
    got = run(mc, ma, mb, ext, A, B, alpha, beta, C)
    np.testing.assert_allclose(got.out64, ref, rtol=1e-12, atol=1e-12)


# ------------------------------------------------------------- GEMM case ---

def gemm_by_definition(A, B, C, alpha, beta):
    """Listing 1: the naive triple loop, C_ij = alpha * sum_k A_ik B_kj + beta C_ij."""
    M, K = A.shape
    N = B.shape[1]
    out = np.empty((M, N))
    for j in range(N):
        for i in range(M):
            tmp = 0.0
            for k in range(K):
                tmp += float(A[i, k]) * float(B[k, j])
            out[i, j] = alpha * tmp + (beta * float(C[i, j]) if beta != 0 else 0.0)
    return out


@pytest.mark.parametrize("M,N,K", [(7, 5, 3), (16, 9, 11), (1, 4, 6), (5, 1, 1)])
@pytest.mark.parametrize("beta", [0.0, 0.5])
def test_gemm_by_definition(M, N, K, beta):
    """When |I_m| = |I_n| = |I_k| = 1 the contraction is a GEMM (Sec. 2.2 example)."""
    rng = np.random.default_rng(M * 100 + N * 10 + K)
    A, B, C = rand(rng, (M, K)), rand(rng, (K, N)), rand(rng, (M, N))
    ext = {"m1": M, "n1": N, "k1": K}
    got = run("m1,n1", "m1,k1", "k1,n1", ext, A, B, -1.5, beta, C)
    np.testing.assert_allclose(got.out64, gemm_by_definition(A, B, C, -1.5, beta),
                               rtol=1e-13, atol=1e-13)
    np.testing.assert_allclose(got.out64, -1.5 * (A @ B) + beta * C, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("case", ["NN", "TN", "NT", "TT"])
def test_gemm_transposes_matmul(case):
    """Transposed storage is just another mode order: compare with numpy.matmul."""
    rng = np.random.default_rng(7)
    M, N, K = 33, 17, 29
    A = rand(rng, (M, K)) if case[0] == "N" else rand(rng, (K, M))
    B = rand(rng, (K, N)) if case[1] == "N" else rand(rng, (N, K))
    ma = "m,k" if case[0] == "N" else "k,m"
    mb = "k,n" if case[1] == "N" else "n,k"
    got = run("m,n", ma, mb, {"m": M, "n": N, "k": K}, A, B)
    Am = A if case[0] == "N" else A.T
    Bm = B if case[1] == "N" else B.T
    np.testing.assert_allclose(got.out64, Am @ Bm, rtol=1e-12, atol=1e-12)


# ----------------------------------------------------------- closed forms ---

def test_all_ones_gives_contracted_size():
    """A = B = 1: every element is alpha * S_Ik + beta * C_in."""
    ext = {"a": 3, "b": 4, "c": 2, "e": 5, "f": 3}
    A = np.ones((5, 3, 3), order="F")      # e, a, f
    B = np.ones((4, 3, 2, 5), order="F")   # b, f, c, e
    C = np.asfortranarray(np.random.default_rng(0).uniform(-1, 1, (3, 4, 2)))
    got = run("a,b,c", "e,a,f", "b,f,c,e", ext, A, B, 2.0, -1.0, C)
    np.testing.assert_allclose(got.out64, 2.0 * 15 - C, rtol=0, atol=1e-14)


def test_kronecker_delta_gives_transposition():
    """B = delta between I_k and I_n turns the contraction into the general
    transposition of Eq. 4: C_{Pi(i..)} = alpha * A_{i..} + beta * C."""
    rng = np.random.default_rng(3)
    ext = {"i": 4, "j": 3, "k": 5, "p": 4, "q": 3}
    A = rand(rng, (4, 3))          # A[i, j]   (i, j contracted)
    # B[p, i, q, j] = delta(p,i) delta(q,j): C[q, p] = sum_{i,j} A[i,j] B[p,i,q,j] = A[p, q]
    B = np.zeros((4, 4, 3, 3), order="F")
    for p in range(4):
        for q in range(3):
            B[p, p, q, q] = 1.0
    C = rand(rng, (3, 4))
    got = run("q,p", "i,j", "p,i,q,j", ext, A, B, 0.5, 2.0, C)
    np.testing.assert_allclose(got.out64, 0.5 * A.T + 2.0 * C, rtol=0, atol=1e-15)


def test_beta_zero_does_not_read_c():
    """beta == 0: C is an output only, NaN in C must not propagate."""
    rng = np.random.default_rng(4)
    A, B = rand(rng, (3, 4)), rand(rng, (4, 2))
    C = np.full((3, 2), np.nan, order="F")
    got = oracle.contract("m,n", "m,k", "k,n", A, B, 1.0, 0.0, C)
    assert np.all(np.isfinite(got.out64))
    np.testing.assert_allclose(got.out64, A @ B, rtol=1e-14)


def test_alpha_zero_does_not_read_operands():
    A = np.full((3, 4), np.nan, order="F")
    B = np.full((4, 2), np.nan, order="F")
    C = rand(np.random.default_rng(5), (3, 2))
    got = oracle.contract("m,n", "m,k", "k,n", A, B, 0.0, 3.0, C)
    np.testing.assert_array_equal(got.out64, 3.0 * C)


def test_zero_extent_is_empty_sum():
    A = np.zeros((3, 0), order="F")
    B = np.zeros((0, 2), order="F")
    C = rand(np.random.default_rng(6), (3, 2))
    got = oracle.contract("m,n", "m,k", "k,n", A, B, 1.0, -2.0, C)
    np.testing.assert_array_equal(got.out64, -2.0 * C)
    np.testing.assert_array_equal(got.den64, 2.0 * np.abs(C))


def test_integer_inputs_are_exact():
    """Integers in [-4, 4]: the fp64 sum is exact, so it equals Python's
    arbitrary-precision integer sum."""
    rng = np.random.default_rng(8)
    ext = {"a": 5, "b": 4, "c": 3, "d": 6, "e": 7}
    A = rand(rng, (7, 5, 6), kind="int")    # e, a, d
    B = rand(rng, (6, 4, 3, 7), kind="int")  # d, b, c, e
    got = run("a,b,c", "e,a,d", "d,b,c,e", ext, A, B)
    Ai, Bi = A.astype(np.int64), B.astype(np.int64)
    for a, b, c in itertools.product(range(5), range(4), range(3)):
        exact = sum(int(Ai[e, a, d]) * int(Bi[d, b, c, e]) for e in range(7) for d in range(6))
        assert got.out64[a, b, c] == exact


# ------------------------------------------------------------ invariances ---

def _int_problem(seed):
    rng = np.random.default_rng(seed)
    mc, ma, mb, ext = wl.random_problem(rng, max_rank=5, max_ext=5)
    sh = lambda m: [ext[x] for x in split(m)]
    return rng, mc, ma, mb, ext, rand(rng, sh(ma), kind="int"), rand(rng, sh(mb), kind="int"), \
        rand(rng, sh(mc), kind="int")


@pytest.mark.parametrize("seed", range(10))
def test_relabelling_is_bit_identical(seed):
    rng, mc, ma, mb, ext, A, B, C = _int_problem(3000 + seed)
    A = A + rand(rng, A.shape) * 0.001   # non-integers: bit-identity is a real check
    names = sorted(ext)
    new = {n: f"r{i}" for i, n in enumerate(rng.permutation(names))}
    ren = lambda m: ",".join(new[x] for x in split(m))
    e2 = {new[k]: v for k, v in ext.items()}
    g1 = run(mc, ma, mb, ext, A, B, 1.5, 0.5, C)
    g2 = run(ren(mc), ren(ma), ren(mb), e2, A, B, 1.5, 0.5, C)
    np.testing.assert_array_equal(g1.out64, g2.out64)


@pytest.mark.parametrize("seed", range(10))
def test_storage_permutation_and_operand_swap(seed):
    """Permuting A's physical storage (with the matching mode string), swapping
    A and B, and permuting C's modes give the same values (integer inputs, so
    the summation order cannot matter)."""
    rng, mc, ma, mb, ext, A, B, C = _int_problem(4000 + seed)
    base = run(mc, ma, mb, ext, A, B, 2.0, -1.0, C)
    la = split(ma)
    perm = list(rng.permutation(len(la)))
    A2 = np.asfortranarray(np.transpose(A, perm))
    ma2 = ",".join(la[p] for p in perm)
    np.testing.assert_array_equal(run(mc, ma2, mb, ext, A2, B, 2.0, -1.0, C).out64, base.out64)
    np.testing.assert_array_equal(run(mc, mb, ma, ext, B, A, 2.0, -1.0, C).out64, base.out64)
    lc = split(mc)
    pc = list(rng.permutation(len(lc)))
    C2 = np.asfortranarray(np.transpose(C, pc))
    mc2 = ",".join(lc[p] for p in pc)
    got = run(mc2, ma, mb, ext, A, B, 2.0, -1.0, C2)
    np.testing.assert_array_equal(got.out64, np.transpose(base.out64, pc))


def test_linearity_in_alpha_and_beta():
    rng, mc, ma, mb, ext, A, B, C = _int_problem(5000)
    t = run(mc, ma, mb, ext, A, B, 1.0, 0.0, C).out64
    got = run(mc, ma, mb, ext, A, B, -3.0, 0.25, C).out64
    np.testing.assert_array_equal(got, -3.0 * t + 0.25 * C)


# ------------------------------------------------------------------ TTGT ---

@pytest.mark.parametrize("seed", range(8))
def test_ttgt_decomposition(seed):
    """Sec. 4 / Listing 5 candidate 1: unfold A to (I_m, I_k) and B to (I_k, I_n)
    by explicit transpositions, one matmul, fold X back into C's order."""
    rng = np.random.default_rng(6000 + seed)
    mc, ma, mb, ext = wl.random_problem(rng, max_rank=6, max_ext=5)
    lc, la, lb = split(mc), split(ma), split(mb)
    Im = [m for m in la if m in lc]
    In = [m for m in lb if m in lc]
    Ik = [m for m in la if m not in lc]
    A = rand(rng, [ext[m] for m in la])
    B = rand(rng, [ext[m] for m in lb])
    S = lambda I: int(np.prod([ext[m] for m in I])) if I else 1
    At = np.transpose(A, [la.index(m) for m in Im + Ik]).reshape(S(Im), S(Ik), order="F")
    Bt = np.transpose(B, [lb.index(m) for m in Ik + In]).reshape(S(Ik), S(In), order="F")
    X = (At @ Bt).reshape([ext[m] for m in Im + In], order="F")
    Cref = np.transpose(X, [(Im + In).index(m) for m in lc])
    got = run(mc, ma, mb, ext, A, B)
    np.testing.assert_allclose(got.out64, Cref, rtol=1e-12, atol=1e-12)


# ------------------------------------------------- Listing 8 (LoG) code ---

def test_listing8_loops_over_gemm():
    """The paper's generated LoG code for C_abcijk = A_ijmc B_mkab (all 24):
    a loop over c and k around a GEMM on super-indices (ab) and (ij), with the
    leading dimensions and offsets of Listing 8.  The oracle must agree at
    sampled C elements of the full 24^6 problem."""
    g = json.load(open(os.path.join(GOLDEN, "listing8_log.json")))
    n = g["contraction"]["extent"]
    rng = np.random.default_rng(88)
    A = rng.uniform(-1, 1, n ** 4)   # flat column-major storage of A[i,j,m,c]
    B = rng.uniform(-1, 1, n ** 4)   # flat column-major storage of B[m,k,a,b]
    m_, n_, k_ = g["gemm"]["m"], g["gemm"]["n"], g["gemm"]["k"]
    lda, ldb, ldc = g["leading_dims"]["lda_on_B"], g["leading_dims"]["ldb_on_A"], \
        g["leading_dims"]["ldc"]
    off = g["offsets"]
    for (c, k) in [(0, 0), (5, 17), (23, 23)]:
        # sgemm("T","T", m_, n_, k_, 1, &B[k*24], lda, &A[c*13824], ldb, 0, &C[...], ldc)
        opB = np.lib.stride_tricks.as_strided(B[k * off["B_per_k"]:], (k_, m_),
                                              (8, 8 * lda))        # B block (k_ x m_), col-major
        opA = np.lib.stride_tricks.as_strided(A[c * off["A_per_c"]:], (n_, k_),
                                              (8, 8 * ldb))        # A block (n_ x k_), col-major
        X = opB.T @ opA.T                                           # (m_ x n_) = C_{(ab),(ij)}
        cbase = c * off["C_per_c"] + k * off["C_per_k"]
        rows = rng.integers(0, m_, 64)
        cols = rng.integers(0, n_, 64)
        pts = cbase + rows + cols * ldc                             # linear positions in C
        Af = A.reshape(n, n, n, n, order="F")
        Bf = B.reshape(n, n, n, n, order="F")
        res = oracle.contract("abcijk", "ijmc", "mkab", Af, Bf, shape_C=[n] * 6, points=pts)
        np.testing.assert_allclose(res.out64, X[rows, cols], rtol=1e-12, atol=1e-12)
    assert m_ == g["super_indices"]["ab"] and n_ == g["super_indices"]["ij"] and k_ == n
    assert lda == n * n and ldb == n * n and ldc == n * n * n


# ----------------------------------------------------- index-set examples ---

def test_paper_index_set_examples():
    """Every contraction the paper states with its index sets is accepted and
    agrees with einsum (so the classification the oracle uses is the paper's)."""
    cases = json.load(open(os.path.join(GOLDEN, "index_sets.json")))["cases"]
    rng = np.random.default_rng(9)
    for cs in cases:
        names = set(split(cs["C"])) | set(split(cs["A"])) | set(split(cs["B"]))
        ext = {m: int(rng.integers(2, 4)) for m in names}
        lc, la = split(cs["C"]), split(cs["A"])
        # the sets, by the definition of Sec. 2.2
        assert sorted(m for m in la if m in lc) == sorted(cs["I_m"])
        assert sorted(m for m in la if m not in lc) == sorted(cs["I_k"])
        A = rand(rng, [ext[m] for m in la])
        B = rand(rng, [ext[m] for m in split(cs["B"])])
        got = run(cs["C"], cs["A"], cs["B"], ext, A, B)
        ref = einsum_ref(cs["C"], cs["A"], cs["B"], A, B, 1.0, 0.0, None)
        np.testing.assert_allclose(got.out64, ref, rtol=1e-12, atol=1e-12)


# ------------------------------------------------------------ error paths ---

@pytest.mark.parametrize("mc,ma,mb", [
    ("m,n,b", "m,k,b", "k,n,b"),   # b in all three tensors (Sec. 2.2 fn. 9)
    ("m,n", "m,k", "n"),           # k only in A
    ("m,n,z", "m,k", "k,n"),       # z only in C
    ("m,n", "m,m,k", "k,n"),       # repeated index
    ("m,n", "m,,k", "k,n"),        # empty name
])
def test_invalid_indices_rejected(mc, ma, mb):
    A = np.zeros([2] * len(split(ma)), order="F")
    B = np.zeros([2] * len(split(mb)), order="F")
    with pytest.raises(oracle.OracleError):
        oracle.contract(mc, ma, mb, A, B, shape_C=[2] * len(split(mc)))


def test_extent_mismatch_rejected():
    A = np.zeros((2, 3), order="F")
    B = np.zeros((4, 2), order="F")
    with pytest.raises(oracle.OracleError):
        oracle.contract("m,n", "m,k", "k,n", A, B, shape_C=[2, 2])


# ------------------------------------------------------ flop-count formula ---

def test_flop_counts_of_workloads():
    """Eq. 14's numerator 2 * S_Im * S_In * S_Ik for the five workloads."""
    expect = {1: 2 * 1024 * 32 * 32, 2: 2 * 12544 * 12544 * 16, 3: 2 * 2304 ** 3,
              4: 2 * 13824 * 13824 * 24, 5: 2 * 4096 ** 3}
    for w in wl.WORKLOADS:
        assert wl.flop_count(w) == expect[w.number]


def test_error_metric_catches_a_dropped_term():
    """The relative-error measure flags a result that misses one product."""
    rng = np.random.default_rng(10)
    A, B = rand(rng, (8, 16)), rand(rng, (16, 8))
    ref = oracle.contract("m,n", "m,k", "k,n", A, B, shape_C=[8, 8])
    bad = A[:, :15] @ B[:15, :]
    assert oracle.rel_error(bad, ref) > 1e-3
    assert oracle.rel_error(A @ B, ref) < 1e-14


# ------------------------------- the parity metric's denominator (den64) ---
#
# The parity bar divides |GPU - out64| by den64 = |alpha| sum_k |a||b| +
# |beta| |c|: the benchmark spec's metric max|diff| / sum_k |A||B| (Sec. 2.2, Eq. 3
# with its alpha and beta).  These checks fix den64 independently of the
# oracle's own loop: closed forms, a hand computation and invariants that a
# dropped term, a signed instead of absolute factor, or a missing |alpha| /
# |beta| would break.

def signs(rng, shape):
    """Entries +1 or -1 with random sign: |a| = 1 everywhere."""
    return np.asfortranarray(rng.choice([-1.0, 1.0], size=shape))


@pytest.mark.parametrize("seed", range(12))
def test_den_of_unit_magnitudes_is_contracted_size(seed):
    """|a| = |b| = 1 makes sum_k |a||b| = S_Ik exactly, whatever the signs:
    den64 = |alpha| * S_Ik + |beta| * |c|, for either sign of alpha and beta
    and any mode pattern (strided and permuted views included)."""
    rng = np.random.default_rng(4000 + seed)
    mc, ma, mb, ext = wl.random_problem(rng, max_rank=6, max_ext=4,
                                        allow_empty_sets=(seed % 4 == 3))
    sk = int(np.prod([ext[m] for m in split(ma) if m not in split(mc)]))
    A = signs(rng, [ext[m] for m in split(ma)])
    B = signs(rng, [ext[m] for m in split(mb)])
    if seed % 2:   # a strided view of B
        big = signs(rng, [2 * ext[m] for m in split(mb)])
        B = big[tuple(slice(0, None, 2) for _ in split(mb))]
    alpha = [1.5, -0.75, -2.0, 0.5][seed % 4]
    beta = [0.0, -1.25, 2.0][seed % 3]
    C = rand(rng, [ext[m] for m in split(mc)]) if beta != 0 else None
    got = run(mc, ma, mb, ext, A, B, alpha, beta, C)
    expect = abs(alpha) * sk + (abs(beta) * np.abs(C) if beta != 0 else 0.0)
    np.testing.assert_array_equal(got.den64, np.broadcast_to(expect, got.den64.shape))


def test_den_hand_computed_2x2x2():
    """C[m,n] = alpha * A[m,k] B[k,n] + beta * C[m,n] with m, n, k of extent 2,
    worked by hand:
        A = [[1, -2], [3, -4]] (rows m, columns k), B = [[-1, 0.5], [2, -3]]
        (rows k, columns n), C = [[1, -1], [2, -2]], alpha = -2, beta = -0.5.
        sum_k |a||b|: (0,0) 1+4 = 5, (0,1) 0.5+6 = 6.5, (1,0) 3+8 = 11,
                      (1,1) 1.5+12 = 13.5
        den = 2 * that + 0.5 * |c| = 10.5, 13.5, 23, 28
        sum_k ab:     -5, 6.5, -11, 13.5
        out = -2 * that - 0.5 * c = 9.5, -12.5, 21, -26."""
    A = np.array([[1.0, -2.0], [3.0, -4.0]], order="F")
    B = np.array([[-1.0, 0.5], [2.0, -3.0]], order="F")
    C = np.array([[1.0, -1.0], [2.0, -2.0]], order="F")
    got = oracle.contract("m,n", "m,k", "k,n", A, B, -2.0, -0.5, C)
    np.testing.assert_array_equal(got.den64, [[10.5, 13.5], [23.0, 28.0]])
    np.testing.assert_array_equal(got.out64, [[9.5, -12.5], [21.0, -26.0]])


@pytest.mark.parametrize("seed", range(6))
def test_den_bounds_the_result_and_ignores_signs(seed):
    """Triangle inequality: |out64| <= den64 element by element, and den64 >= 0.
    Flipping the sign of any entries of A, B or C leaves den64 bit-identical
    (|-x| = |x| exactly, the same summation order), while out64 changes."""
    rng = np.random.default_rng(4100 + seed)
    mc, ma, mb, ext = wl.random_problem(rng, max_rank=6, max_ext=5)
    shp = lambda m: [ext[x] for x in split(m)]
    A, B, C = rand(rng, shp(ma)), rand(rng, shp(mb)), rand(rng, shp(mc))
    alpha, beta = (-1.5, -0.5) if seed % 2 else (0.75, 2.0)
    r = run(mc, ma, mb, ext, A, B, alpha, beta, C)
    assert np.all(r.den64 >= 0)
    assert np.all(np.abs(r.out64) <= r.den64 * (1 + 1e-15))
    flip = lambda X: np.asfortranarray(X * rng.choice([-1.0, 1.0], size=X.shape))
    r2 = run(mc, ma, mb, ext, flip(A), flip(B), alpha, beta, flip(C))
    np.testing.assert_array_equal(r2.den64, r.den64)
    # powers of two scale exactly: den(2 alpha, 2 beta) = 2 den(alpha, beta)
    r3 = run(mc, ma, mb, ext, A, B, 2 * alpha, 2 * beta, C)
    np.testing.assert_array_equal(r3.den64, 2 * r.den64)


def test_rel_error_refuses_a_negative_or_nan_denominator():
    """A negative (or NaN) den64 would make every check pass vacuously."""
    ref = oracle.Result(np.array([1.0, 2.0]), np.array([1.0, -1.0]))
    with pytest.raises(ValueError):
        oracle.rel_error(np.array([1.0, 2.0]), ref)
    ref = oracle.Result(np.array([1.0, 2.0]), np.array([1.0, np.nan]))
    with pytest.raises(ValueError):
        oracle.rel_error(np.array([1.0, 2.0]), ref)
    ref = oracle.Result(np.array([1.0, 2.0]), np.array([1.0, 1.0]))
    with pytest.raises(ValueError):
        oracle.rel_error(np.array([1.0, 2.0, 3.0]), ref)   # sizes differ


# ------------------------------------------- Eq. 4: tensor transposition ---

def test_transpose_worked_example():
    """A 2x3 matrix 1..6 in Fortran order, transposed (Sec. 2.3 with d = 2):
    rows become columns."""
    A = np.arange(1, 7, dtype=np.float64).reshape(2, 3, order="F")   # [[1,3,5],[2,4,6]]
    r = oracle.transpose(A, [1, 0])
    assert r.out64.shape == (3, 2)
    assert r.out64.tolist() == [[1.0, 2.0], [3.0, 4.0], [5.0, 6.0]]


@pytest.mark.parametrize("dtype", [np.float32, np.float64])
def test_transpose_matches_numpy_axis_permutation(dtype):
    """Output mode j is input mode perm[j]: numpy's transpose with the same
    axes gives the same array (alpha 1, beta 0, exact)."""
    rng = np.random.default_rng(7)
    for perm in ([0, 1, 2], [2, 0, 1], [1, 2, 0], [2, 1, 0], [3, 1, 0, 2]):
        shape = [2, 3, 4, 5][:len(perm)]
        A = rng.standard_normal(shape).astype(dtype)
        got = oracle.transpose(A, perm).out64
        assert np.array_equal(got, np.transpose(A, perm).astype(np.float64))


def test_transpose_cycle_is_not_its_inverse():
    """A 3-cycle distinguishes perm from its inverse (a swapped convention
    would fail here)."""
    A = np.arange(24, dtype=np.float64).reshape(2, 3, 4)
    got = oracle.transpose(A, [1, 2, 0]).out64
    assert got.shape == (3, 4, 2)
    for i, j, k in itertools.product(range(2), range(3), range(4)):
        assert got[j, k, i] == A[i, j, k]
    inverse = oracle.transpose(A, [2, 0, 1]).out64
    assert inverse.shape == (4, 2, 3)


def test_transpose_round_trip_restores_input():
    rng = np.random.default_rng(8)
    A = rng.standard_normal((3, 4, 2, 5))
    perm = [2, 0, 3, 1]
    inv = list(np.argsort(perm))
    once = oracle.transpose(A, perm).out64
    back = oracle.transpose(np.asfortranarray(once), inv).out64
    assert np.array_equal(back, A)


def test_transpose_scaling_closed_form():
    """Identity permutation: Eq. 4 reduces to alpha * a + beta * b elementwise
    (BLAS axpby); den = |alpha a| + |beta b|."""
    rng = np.random.default_rng(9)
    A = rng.standard_normal((4, 5))
    B = rng.standard_normal((4, 5))
    r = oracle.transpose(A, [0, 1], alpha=0.5, beta=-2.0, B=B)
    assert np.array_equal(r.out64, 0.5 * A + -2.0 * B)
    assert np.array_equal(r.den64, np.abs(0.5 * A) + np.abs(-2.0 * B))


def test_transpose_strided_views_and_beta():
    """Strided input and a strided old output, beta != 0, against numpy."""
    rng = np.random.default_rng(10)
    base = rng.standard_normal((7, 9, 6))
    A = base[::2, 1::2, :5]                      # (4, 4, 5), gaps in every mode
    perm = [2, 0, 1]
    obase = rng.standard_normal((11, 10, 9))
    B = obase[1:6, :8:2, 2:6]                    # (5, 4, 4) = A.shape[perm], gapped
    assert list(B.shape) == [A.shape[p] for p in perm]
    r = oracle.transpose(A, perm, alpha=1.5, beta=0.25, B=B)
    ref = 1.5 * np.transpose(A, perm) + 0.25 * B
    assert np.allclose(r.out64, ref, rtol=0, atol=1e-15)


def test_transpose_beta_zero_ignores_old_output():
    A = np.ones((2, 2))
    r = oracle.transpose(A, [1, 0], alpha=3.0, beta=0.0, B=None)
    assert np.array_equal(r.out64, 3.0 * np.ones((2, 2)))


def test_transpose_rejects_bad_permutation():
    A = np.ones((2, 3))
    for perm in ([0, 0], [0, 2], [1]):
        with pytest.raises((oracle.OracleError, IndexError, ValueError)):
            oracle.transpose(A, perm)


def test_transpose_empty_and_scalar():
    A = np.ones((0, 3))
    assert oracle.transpose(A, [1, 0]).out64.shape == (3, 0)
    s = np.array(2.5)
    assert float(oracle.transpose(s, [], alpha=2.0).out64) == 5.0
