/*
 * gett_oracle.c -- plain CPU definition of the dense tensor contraction
 *
 *     C_{Pi_C(I_m u I_n)} <- alpha * A_{Pi_A(I_m u I_k)} * B_{Pi_B(I_n u I_k)}
 *                            + beta * C_{Pi_C(I_m u I_n)}
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the correctness reference for the
 * GPU library: only the test suite, the smoke check and the CPU baseline leg
 * of the benchmark load it.  It shares no code, header or table with the GPU
 * path, and the GPU path never calls it.
 *
 * What it computes (paper Sec. 2.2, Eq. 2 and Eq. 3; the naive loop nest of
 * Listing 3 in Sec. 3, which the paper itself uses as its correctness
 * reference in Sec. 7):
 *   - index sets (Sec. 2.2): I_m = free indices that appear in A and C,
 *     I_n = free indices that appear in B and C, I_k = contracted indices
 *     that appear in A and B but not in C.  An index present in all three
 *     tensors is not a contraction of this form (Sec. 2.2, footnote 9) and is
 *     rejected, as is an index present in only one tensor or twice in one.
 *   - for every element x of C:
 *         t(x)   = sum over the multi-index y of I_k of A[x_m, y] * B[y, x_n]
 *         out(x) = alpha * t(x) + beta * C_in(x)
 *     The beta term is added once, after the sum (Listing 1, Listing 3,
 *     Eq. 3, Eq. 11); Eq. 1 and Eq. 2 print it inside the sum, which is read
 *     as the same operation.  When beta == 0 the C input is not read (BLAS
 *     convention; the paper is silent).
 *   - memory layout: every tensor is addressed through one stride per mode,
 *     in elements; the default in the paper is the Fortran layout (Sec. 2.2),
 *     which callers express as column-major strides.
 *   - arithmetic: every product and every partial sum is formed in IEEE
 *     double precision; fp32 inputs are widened exactly.  No rounding to the
 *     output type happens here: callers compare against the unrounded value.
 *   - den(x) = |alpha| * sum_y |A[x_m,y]| * |B[y,x_n]| + |beta| * |C_in(x)| is
 *     returned beside out(x) as the scale of the rounding error.
 *
 * Loop order: C elements are independent; each is computed alone.  The sum
 * over I_k runs as an odometer over the contracted modes in the order they
 * appear in A, with A's first contracted mode varying fastest.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define OR_MAX_MODES 32
#define OR_MAX_NAME 31

enum {
    OR_OK = 0,
    OR_ERR_VALUE = -1,   /* null pointer, bad dtype, negative extent, ... */
    OR_ERR_PARSE = -2,   /* malformed mode string */
    OR_ERR_INDEX = -3,   /* index in 1 or 3 tensors, repeated, extent mismatch */
    OR_ERR_RANGE = -4    /* point index outside C */
};

typedef struct {
    int n;
    char name[OR_MAX_MODES][OR_MAX_NAME + 1];
} or_modes;

/* Mode strings: comma separated names ("m1,k1,m2"; a trailing comma marks a
 * single name, "m1,"), or, with no comma, one character per mode ("akc").
 * Spaces are ignored.  The empty string is a scalar (no modes). */
static int or_parse(const char *s, or_modes *out)
{
    out->n = 0;
    if (!s) return OR_ERR_VALUE;
    int has_comma = strchr(s, ',') != NULL;
    const char *p = s;
    if (!has_comma) {
        for (; *p; ++p) {
            if (*p == ' ') continue;
            if (out->n >= OR_MAX_MODES) return OR_ERR_PARSE;
            out->name[out->n][0] = *p;
            out->name[out->n][1] = 0;
            out->n++;
        }
        return OR_OK;
    }
    while (1) {
        char buf[OR_MAX_NAME + 1];
        int len = 0;
        while (*p && *p != ',') {
            if (*p != ' ') {
                if (len >= OR_MAX_NAME) return OR_ERR_PARSE;
                buf[len++] = *p;
            }
            ++p;
        }
        if (len == 0) {
            if (*p == 0 && out->n > 0) break; /* one trailing comma is allowed */
            return OR_ERR_PARSE;
        }
        if (out->n >= OR_MAX_MODES) return OR_ERR_PARSE;
        buf[len] = 0;
        memcpy(out->name[out->n], buf, (size_t)len + 1);
        out->n++;
        if (*p == 0) break;
        ++p; /* skip comma */
    }
    return OR_OK;
}

static int or_find(const or_modes *m, const char *name)
{
    for (int i = 0; i < m->n; ++i)
        if (strcmp(m->name[i], name) == 0) return i;
    return -1;
}

/* The contraction after classification.  For each C mode: which set it is in
 * and where it sits in A (I_m) or B (I_n).  For each contracted mode, in A's
 * order: its extent and its strides in A and B. */
typedef struct {
    int nc;
    int64_t extC[OR_MAX_MODES];
    int64_t strC[OR_MAX_MODES];
    int64_t strA_of_c[OR_MAX_MODES]; /* stride in A if the C mode is in I_m, else 0 */
    int64_t strB_of_c[OR_MAX_MODES]; /* stride in B if the C mode is in I_n, else 0 */
    int nk;
    int64_t extK[OR_MAX_MODES];
    int64_t strAk[OR_MAX_MODES];
    int64_t strBk[OR_MAX_MODES];
    int64_t sizeC; /* product of C extents */
} or_problem;

static int or_setup(or_problem *P,
                    const char *modesC, const int64_t *extC, const int64_t *strC,
                    const char *modesA, const int64_t *extA, const int64_t *strA,
                    const char *modesB, const int64_t *extB, const int64_t *strB)
{
    or_modes mc, ma, mb;
    int rc;
    if ((rc = or_parse(modesC, &mc)) != OR_OK) return rc;
    if ((rc = or_parse(modesA, &ma)) != OR_OK) return rc;
    if ((rc = or_parse(modesB, &mb)) != OR_OK) return rc;
    if ((mc.n && (!extC || !strC)) || (ma.n && (!extA || !strA)) || (mb.n && (!extB || !strB)))
        return OR_ERR_VALUE;

    /* no repeated index inside one tensor */
    const or_modes *all[3] = {&mc, &ma, &mb};
    for (int t = 0; t < 3; ++t)
        for (int i = 0; i < all[t]->n; ++i)
            for (int j = i + 1; j < all[t]->n; ++j)
                if (strcmp(all[t]->name[i], all[t]->name[j]) == 0) return OR_ERR_INDEX;
    for (int i = 0; i < mc.n; ++i) if (extC[i] < 0) return OR_ERR_VALUE;
    for (int i = 0; i < ma.n; ++i) if (extA[i] < 0) return OR_ERR_VALUE;
    for (int i = 0; i < mb.n; ++i) if (extB[i] < 0) return OR_ERR_VALUE;

    memset(P, 0, sizeof(*P));
    P->nc = mc.n;
    P->sizeC = 1;
    /* every C mode must be in exactly one of A, B (I_m or I_n) */
    for (int i = 0; i < mc.n; ++i) {
        int ia = or_find(&ma, mc.name[i]);
        int ib = or_find(&mb, mc.name[i]);
        if ((ia >= 0) == (ib >= 0)) return OR_ERR_INDEX; /* in both (fn. 9) or in neither */
        P->extC[i] = extC[i];
        P->strC[i] = strC[i];
        if (ia >= 0) {
            if (extA[ia] != extC[i]) return OR_ERR_INDEX;
            P->strA_of_c[i] = strA[ia];
        } else {
            if (extB[ib] != extC[i]) return OR_ERR_INDEX;
            P->strB_of_c[i] = strB[ib];
        }
        P->sizeC *= extC[i];
    }
    /* every A mode not in C must be in B (I_k) */
    for (int i = 0; i < ma.n; ++i) {
        if (or_find(&mc, ma.name[i]) >= 0) continue;
        int ib = or_find(&mb, ma.name[i]);
        if (ib < 0) return OR_ERR_INDEX;
        if (extB[ib] != extA[i]) return OR_ERR_INDEX;
        P->extK[P->nk] = extA[i];
        P->strAk[P->nk] = strA[i];
        P->strBk[P->nk] = strB[ib];
        P->nk++;
    }
    /* every B mode must be in C or in A */
    for (int i = 0; i < mb.n; ++i)
        if (or_find(&mc, mb.name[i]) < 0 && or_find(&ma, mb.name[i]) < 0) return OR_ERR_INDEX;
    return OR_OK;
}

static inline double or_load(int dtype, const void *p, int64_t off)
{
    return dtype == 0 ? (double)((const float *)p)[off] : ((const double *)p)[off];
}

/* One element of C, given its position in C's column-major logical order. */
static void or_element(const or_problem *P, int dtype, double alpha, const void *A,
                       const void *B, double beta, const void *Cin, int64_t lin,
                       double *out, double *den)
{
    int64_t offA = 0, offB = 0, offC = 0;
    int64_t rem = lin;
    for (int i = 0; i < P->nc; ++i) {
        int64_t idx = rem % P->extC[i];
        rem /= P->extC[i];
        offA += idx * P->strA_of_c[i];
        offB += idx * P->strB_of_c[i];
        offC += idx * P->strC[i];
    }
    double acc = 0.0, acc_abs = 0.0;
    int64_t sizeK = 1;
    for (int j = 0; j < P->nk; ++j) sizeK *= P->extK[j];
    if (sizeK > 0 && alpha != 0.0) {
        int64_t cnt[OR_MAX_MODES];
        for (int j = 0; j < P->nk; ++j) cnt[j] = 0;
        int64_t oa = offA, ob = offB;
        for (int64_t y = 0; y < sizeK; ++y) {
            double a = or_load(dtype, A, oa);
            double b = or_load(dtype, B, ob);
            acc += a * b;
            acc_abs += fabs(a) * fabs(b);
            /* advance the odometer: first contracted mode of A fastest */
            for (int j = 0; j < P->nk; ++j) {
                cnt[j]++;
                oa += P->strAk[j];
                ob += P->strBk[j];
                if (cnt[j] < P->extK[j]) break;
                oa -= cnt[j] * P->strAk[j];
                ob -= cnt[j] * P->strBk[j];
                cnt[j] = 0;
            }
        }
    }
    double r = alpha * acc;
    double d = fabs(alpha) * acc_abs;
    if (beta != 0.0) {
        double c = or_load(dtype, Cin, offC);
        r += beta * c;
        d += fabs(beta) * fabs(c);
    }
    *out = r;
    *den = d;
}

/*
 * oracle_contract: compute out64 / den64 for C elements.
 *   dtype    0 = float32, 1 = float64 (type of A, B and C_in)
 *   modes*   mode strings; ext* extents per mode; str* strides per mode (elements)
 *   A, B     operands (not read when alpha == 0 or the contracted size is 0)
 *   Cin      input C (not read when beta == 0; may then be NULL)
 *   npts     number of C elements to compute; pts their positions in C's
 *            column-major logical order (mode 0 fastest).  pts == NULL means
 *            every element, npts must then be the size of C.
 *   out64, den64  npts doubles each
 *   nthreads OpenMP threads (<= 0: runtime default)
 * Returns 0 or a negative OR_ERR_* code.
 */
int oracle_contract(int dtype,
                    const char *modesC, const int64_t *extC, const int64_t *strC,
                    const char *modesA, const int64_t *extA, const int64_t *strA,
                    const char *modesB, const int64_t *extB, const int64_t *strB,
                    double alpha, const void *A, const void *B, double beta,
                    const void *Cin, int64_t npts, const int64_t *pts,
                    double *out64, double *den64, int nthreads)
{
    if (dtype != 0 && dtype != 1) return OR_ERR_VALUE;
    or_problem P;
    int rc = or_setup(&P, modesC, extC, strC, modesA, extA, strA, modesB, extB, strB);
    if (rc != OR_OK) return rc;
    if (npts < 0 || (npts > 0 && (!out64 || !den64))) return OR_ERR_VALUE;
    if (!pts && npts != P.sizeC) return OR_ERR_VALUE;
    if (beta != 0.0 && npts > 0 && !Cin) return OR_ERR_VALUE;
    if (alpha != 0.0 && npts > 0 && (!A || !B)) return OR_ERR_VALUE;
    if (pts)
        for (int64_t p = 0; p < npts; ++p)
            if (pts[p] < 0 || pts[p] >= P.sizeC) return OR_ERR_RANGE;
#ifdef _OPENMP
    if (nthreads <= 0) nthreads = omp_get_max_threads();
#pragma omp parallel for schedule(dynamic, 256) num_threads(nthreads)
#endif
    for (int64_t p = 0; p < npts; ++p) {
        int64_t lin = pts ? pts[p] : p;
        or_element(&P, dtype, alpha, A, B, beta, Cin, lin, &out64[p], &den64[p]);
    }
    (void)nthreads;
    return OR_OK;
}

/* Number of threads the OpenMP runtime would use by default. */
int oracle_max_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/*
 * oracle_transpose: the general tensor transposition with input and output
 * scaling of Sec. 2.3, Eq. 4:
 *
 *     out[Pi(i_1, ..., i_d)] = alpha * in[i_1, ..., i_d] + beta * out_in[Pi(i_1, ..., i_d)]
 *
 *   dtype    0 = float32, 1 = float64 (type of in and out_in)
 *   rank     d (0 <= d <= 32); ext[d] extents of `in`; str_in[d] its strides
 *   perm     output mode j is input mode perm[j] (a permutation of 0..d-1)
 *   in       not read when alpha == 0
 *   out_in   the old output (not read when beta == 0), addressed by
 *            str_out_in[j] for output mode j
 *   out64, den64  dense column-major over the output's extents
 *            (ext[perm[0]] fastest): the unrounded fp64 result and
 *            |alpha * in| + |beta * out_in| as the scale of its rounding error.
 * Every input element is visited once, by an odometer over the input modes
 * (mode 0 fastest); its output position is recomputed from the multi-index.
 */
int oracle_transpose(int dtype, int rank, const int64_t *ext, const int64_t *str_in,
                     const int64_t *perm, double alpha, const void *in, double beta,
                     const void *out_in, const int64_t *str_out_in, double *out64, double *den64)
{
    if (dtype != 0 && dtype != 1) return OR_ERR_VALUE;
    if (rank < 0 || rank > OR_MAX_MODES) return OR_ERR_VALUE;
    int seen[OR_MAX_MODES];
    for (int j = 0; j < rank; ++j) seen[j] = 0;
    for (int j = 0; j < rank; ++j) {
        if (perm[j] < 0 || perm[j] >= rank || seen[perm[j]]) return OR_ERR_VALUE;
        seen[perm[j]] = 1;
    }
    int64_t size = 1;
    for (int i = 0; i < rank; ++i) {
        if (ext[i] < 0) return OR_ERR_VALUE;
        size *= ext[i];
    }
    if (size == 0) return OR_OK;
    if ((alpha != 0.0 && !in) || (beta != 0.0 && !out_in) || !out64 || !den64)
        return OR_ERR_VALUE;
    /* dense column-major stride of each output mode, then of each input mode */
    int64_t dense_out[OR_MAX_MODES], pos_stride[OR_MAX_MODES], old_stride[OR_MAX_MODES];
    int64_t acc = 1;
    for (int j = 0; j < rank; ++j) {
        dense_out[j] = acc;
        acc *= ext[perm[j]];
    }
    for (int j = 0; j < rank; ++j) {
        pos_stride[perm[j]] = dense_out[j];
        old_stride[perm[j]] = str_out_in ? str_out_in[j] : 0;
    }
    int64_t idx[OR_MAX_MODES];
    for (int i = 0; i < rank; ++i) idx[i] = 0;
    for (int64_t n = 0; n < size; ++n) {
        int64_t offIn = 0, pos = 0, offOld = 0;
        for (int i = 0; i < rank; ++i) {
            offIn += idx[i] * str_in[i];
            pos += idx[i] * pos_stride[i];
            offOld += idx[i] * old_stride[i];
        }
        double r = 0.0, d = 0.0;
        if (alpha != 0.0) {
            double a = or_load(dtype, in, offIn);
            r = alpha * a;
            d = fabs(alpha * a);
        }
        if (beta != 0.0) {
            double b = or_load(dtype, out_in, offOld);
            r += beta * b;
            d += fabs(beta * b);
        }
        out64[pos] = r;
        den64[pos] = d;
        for (int i = 0; i < rank; ++i) {
            if (++idx[i] < ext[i]) break;
            idx[i] = 0;
        }
    }
    return OR_OK;
}
