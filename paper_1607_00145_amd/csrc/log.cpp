// log.cpp -- Loops-over-GEMM (Sec. 5, Listing 7), the second method GETT is
// measured against.
//
// The contraction is cut into 2D slices that an ordinary GEMM can multiply
// in place (one unit-stride dimension per operand, a leading dimension for
// the other), and the remaining indices are looped over:
//   * the stride-one index of A, of B and of C must be among the GEMM's three
//     indices; when C's stride-one index belongs to B, A and B exchange roles
//     so that it becomes the GEMM's m index;
//   * no index set may hold two of those stride-one indices (the slice would
//     need strides in both dimensions): LoG is then not applicable;
//   * a set without a stride-one index contributes its largest index (the
//     selection metric of Sec. 5 is the GEMM's flop count); super-indices
//     merged beforehand count as one index;
//   * the other indices are loops.  All loop orders are equivalent here: the
//     largest free loop index becomes the batch of one strided-batched GEMM
//     call (independent slices of C), the other free loops and the
//     contracted loops are host loops; contracted loops accumulate into the
//     same slice, with beta applied by the first of them only.
#include <hip/hip_runtime_api.h>
#include <rocblas/rocblas.h>
#include <stdint.h>

#include <algorithm>
#include <new>
#include <sstream>
#include <string>
#include <vector>

#include "blas.hpp"
#include "plan.hpp"
#include "transpose.hpp"

namespace gett {
namespace {

struct LoopIdx {
    std::string name;
    int64_t extent;
    int64_t sL, sR, sC;   // strides in the left and right operands and C (0 when absent)
};

}  // namespace
}  // namespace gett

struct gett_log_plan_s {
    gett_dtype_t dtype;
    gett::Analysis an;
    bool swapped = false;                     // left operand is B
    std::string mName, nName, kName;
    int64_t M = 1, N = 1, K = 1;
    bool opL = false, opR = false;            // transposed
    int64_t lda = 1, ldb = 1, ldc = 1;
    bool hasBatch = false;
    gett::LoopIdx batch;
    std::vector<gett::LoopIdx> freeLoops, kLoops;
    int64_t calls = 1;
    std::vector<int64_t> cExt, cStr;
    std::string text;
};

namespace gett {
namespace {

int64_t str_of(const Index &x, int t) { return t == 0 ? x.strC : t == 1 ? x.strA : x.strB; }

// Smallest-stride index of tensor t among the given sets ("" if none).
std::string unit_of(const std::vector<const std::vector<Index> *> &sets, int t)
{
    int64_t best = INT64_MAX;
    std::string n;
    for (auto *s : sets)
        for (auto &x : *s)
            if (str_of(x, t) < best) {
                best = str_of(x, t);
                n = x.name;
            }
    return n;
}

gett_status_t plan_log(gett_log_plan_s &P)
{
    const Analysis &an = P.an;
    // stride-one indices of A, B and C (Listing 7: each tensor's first index)
    const std::string uA = unit_of({&an.Im, &an.Ik}, 1);
    const std::string uB = unit_of({&an.In, &an.Ik}, 2);
    const std::string uC = unit_of({&an.Im, &an.In}, 0);
    bool cInB = false;
    for (auto &x : an.In) cInB |= x.name == uC;
    P.swapped = cInB;
    const int tL = P.swapped ? 2 : 1, tR = P.swapped ? 1 : 2;
    const std::vector<Index> &Im = P.swapped ? an.In : an.Im;
    const std::vector<Index> &In = P.swapped ? an.Im : an.In;
    const std::vector<Index> &Ik = an.Ik;
    auto required = [&](const std::string &n) { return n == uA || n == uB || n == uC; };
    // Pick the GEMM index of one set: its stride-one index, else its largest.
    auto pick = [&](const std::vector<Index> &s, const Index *&out) -> bool {
        out = nullptr;
        int req = 0;
        for (auto &x : s)
            if (required(x.name)) {
                ++req;
                out = &x;
            }
        if (req >= 2) return false;   // two stride-one indices in one set
        if (!out)
            for (auto &x : s)
                if (!out || x.extent > out->extent) out = &x;
        return true;
    };
    const Index *im, *in, *ik;
    if (!pick(Im, im) || !pick(In, in) || !pick(Ik, ik)) return GETT_ERROR_NOT_SUPPORTED;
    // An empty set gives a GEMM dimension of 1.
    auto ext = [](const Index *x) { return x ? x->extent : (int64_t)1; };
    auto stride = [&](const Index *x, int t) { return x ? str_of(*x, t) : (int64_t)1; };
    P.mName = im ? im->name : "";
    P.nName = in ? in->name : "";
    P.kName = ik ? ik->name : "";
    P.M = ext(im);
    P.N = ext(in);
    P.K = ext(ik);
    // Slices: the dimension with unit stride is the GEMM's row dimension.
    auto slice = [](int64_t rows, int64_t sRows, int64_t cols, int64_t sCols, int64_t &ld) -> bool {
        if (rows > 1 && sRows != 1) return false;
        ld = cols > 1 ? sCols : std::max<int64_t>(rows, 1);
        return ld >= std::max<int64_t>(rows, 1);
    };
    // left operand: m x k (op N) or k x m (op T)
    const int64_t sLm = stride(im, tL), sLk = stride(ik, tL);
    if (P.M > 1 && sLm == 1 && slice(P.M, sLm, P.K, sLk, P.lda)) {
        P.opL = false;
    } else if (slice(P.K, sLk, P.M, sLm, P.lda)) {
        P.opL = true;
    } else if (slice(P.M, sLm, P.K, sLk, P.lda)) {
        P.opL = false;
    } else {
        return GETT_ERROR_NOT_SUPPORTED;
    }
    // right operand: k x n (op N) or n x k (op T)
    const int64_t sRk = stride(ik, tR), sRn = stride(in, tR);
    if (P.K > 1 && sRk == 1 && slice(P.K, sRk, P.N, sRn, P.ldb)) {
        P.opR = false;
    } else if (slice(P.N, sRn, P.K, sRk, P.ldb)) {
        P.opR = true;
    } else if (slice(P.K, sRk, P.N, sRn, P.ldb)) {
        P.opR = false;
    } else {
        return GETT_ERROR_NOT_SUPPORTED;
    }
    if (!slice(P.M, stride(im, 0), P.N, stride(in, 0), P.ldc)) return GETT_ERROR_NOT_SUPPORTED;
    for (int64_t v : {P.M, P.N, P.K, P.lda, P.ldb, P.ldc})
        if (v > INT32_MAX) return GETT_ERROR_NOT_SUPPORTED;
    // loops
    auto loop_of = [&](const Index &x) {
        LoopIdx l;
        l.name = x.name;
        l.extent = x.extent;
        l.sL = str_of(x, tL);
        l.sR = str_of(x, tR);
        l.sC = x.strC;
        return l;
    };
    for (auto &x : Im)
        if (&x != im) {
            LoopIdx l = loop_of(x);
            l.sR = 0;
            P.freeLoops.push_back(l);
        }
    for (auto &x : In)
        if (&x != in) {
            LoopIdx l = loop_of(x);
            l.sL = 0;
            P.freeLoops.push_back(l);
        }
    for (auto &x : Ik)
        if (&x != ik) {
            LoopIdx l = loop_of(x);
            l.sC = 0;
            P.kLoops.push_back(l);
        }
    if (!P.freeLoops.empty()) {
        auto it = std::max_element(P.freeLoops.begin(), P.freeLoops.end(),
                                   [](const LoopIdx &a, const LoopIdx &b) { return a.extent < b.extent; });
        P.batch = *it;
        P.hasBatch = true;
        P.freeLoops.erase(it);
        if (P.batch.extent > INT32_MAX) return GETT_ERROR_NOT_SUPPORTED;
    }
    P.calls = 1;
    for (auto &l : P.freeLoops) P.calls *= l.extent;
    for (auto &l : P.kLoops) P.calls *= l.extent;
    return GETT_SUCCESS;
}

void describe(gett_log_plan_s &P)
{
    std::ostringstream o;
    auto loops = [&](const char *key, const std::vector<LoopIdx> &v) {
        o << ",\"" << key << "\":[";
        for (size_t i = 0; i < v.size(); ++i) o << (i ? "," : "") << "\"" << v[i].name << "\"";
        o << "]";
    };
    o << "{\"method\":\"log\",\"dtype\":\"" << (P.dtype == GETT_FLOAT32 ? "f32" : "f64") << "\"";
    o << ",\"swapped\":" << (P.swapped ? "true" : "false");
    o << ",\"gemm\":{\"m_index\":\"" << P.mName << "\",\"n_index\":\"" << P.nName
      << "\",\"k_index\":\"" << P.kName << "\",\"m\":" << P.M << ",\"n\":" << P.N << ",\"k\":" << P.K
      << ",\"op_left\":\"" << (P.opL ? "T" : "N") << "\",\"op_right\":\"" << (P.opR ? "T" : "N")
      << "\",\"lda\":" << P.lda << ",\"ldb\":" << P.ldb << ",\"ldc\":" << P.ldc << "}";
    o << ",\"batch\":";
    if (P.hasBatch)
        o << "{\"index\":\"" << P.batch.name << "\",\"count\":" << P.batch.extent << ",\"stride_left\":"
          << P.batch.sL << ",\"stride_right\":" << P.batch.sR << ",\"stride_c\":" << P.batch.sC << "}";
    else
        o << "null";
    loops("free_loops", P.freeLoops);
    loops("contracted_loops", P.kLoops);
    o << ",\"gemm_calls\":" << P.calls << ",\"empty_c\":" << (P.an.emptyC ? "true" : "false")
      << ",\"empty_sum\":" << (P.an.emptySum ? "true" : "false") << "}";
    P.text = o.str();
}

}  // namespace
}  // namespace gett

extern "C" {

gett_status_t gett_log_plan(gett_log_plan_t *plan, gett_dtype_t dtype, const char *modes_C,
                            const int64_t *extent_C, const int64_t *stride_C, const char *modes_A,
                            const int64_t *extent_A, const int64_t *stride_A, const char *modes_B,
                            const int64_t *extent_B, const int64_t *stride_B)
{
    if (!plan) return GETT_ERROR_INVALID_VALUE;
    *plan = nullptr;
    gett_log_plan_s *p = new (std::nothrow) gett_log_plan_s();
    if (!p) return GETT_ERROR_ALLOC;
    gett_status_t st;
    try {
        int rank[3];
        p->dtype = dtype;
        st = gett::front_end(p->an, dtype, modes_C, extent_C, stride_C, modes_A, extent_A, stride_A,
                             modes_B, extent_B, stride_B, rank, true);
        if (st == GETT_SUCCESS) {
            for (auto *s : {&p->an.Im, &p->an.In})
                for (auto &x : *s) {
                    p->cExt.push_back(x.extent);
                    p->cStr.push_back(x.strC);
                }
            if (!p->an.emptyC && !p->an.emptySum) st = gett::plan_log(*p);
        }
        if (st == GETT_SUCCESS) gett::describe(*p);
    } catch (const std::bad_alloc &) {
        st = GETT_ERROR_ALLOC;
    } catch (...) {
        st = GETT_ERROR_INVALID_VALUE;
    }
    if (st != GETT_SUCCESS) {
        delete p;
        return st;
    }
    *plan = p;
    return GETT_SUCCESS;
}

gett_status_t gett_log_contract(const gett_log_plan_t plan, double alpha, const void *A,
                                const void *B, double beta, void *C, void *stream)
{
    if (!plan) return GETT_ERROR_INVALID_VALUE;
    const gett_log_plan_s &P = *plan;
    if (P.an.emptyC) return GETT_SUCCESS;
    const bool readAB = alpha != 0.0 && !P.an.emptySum;
    if (!gett::operands_ok(P.dtype, P.an, readAB, A, B, C)) return GETT_ERROR_INVALID_VALUE;
    hipStream_t s = (hipStream_t)stream;
    if (!readAB)   // C <- beta * C
        return gett::transpose_launch(P.dtype, (int)P.cExt.size(), P.cExt.data(), P.cStr.data(),
                                      P.cStr.data(), 0.0, nullptr, beta, C, s);
    const int64_t item = P.dtype == GETT_FLOAT32 ? 4 : 8;
    const char *L = static_cast<const char *>(P.swapped ? B : A);
    const char *R = static_cast<const char *>(P.swapped ? A : B);
    char *Cb = static_cast<char *>(C);
    const rocblas_operation ta = P.opL ? rocblas_operation_transpose : rocblas_operation_none;
    const rocblas_operation tb = P.opR ? rocblas_operation_transpose : rocblas_operation_none;
    const rocblas_int m = (rocblas_int)P.M, n = (rocblas_int)P.N, k = (rocblas_int)P.K;
    const rocblas_int lda = (rocblas_int)P.lda, ldb = (rocblas_int)P.ldb, ldc = (rocblas_int)P.ldc;
    const rocblas_int batch = P.hasBatch ? (rocblas_int)P.batch.extent : 1;
    const rocblas_stride bL = P.hasBatch ? P.batch.sL : 0, bR = P.hasBatch ? P.batch.sR : 0,
                         bC = P.hasBatch ? P.batch.sC : 0;
    // odometers over the contracted loops (outer) and the other free loops
    std::vector<int64_t> qk(P.kLoops.size(), 0), qf(P.freeLoops.size(), 0);
    int64_t kOffL = 0, kOffR = 0;
    for (bool firstK = true;; firstK = false) {
        const double be = firstK ? beta : 1.0;
        std::fill(qf.begin(), qf.end(), 0);
        int64_t fOffL = 0, fOffR = 0, fOffC = 0;
        for (;;) {
            const int64_t oL = (kOffL + fOffL) * item, oR = (kOffR + fOffR) * item, oC = fOffC * item;
            const gett_status_t st = gett::with_blas(s, [&](rocblas_handle h) {
                if (P.dtype == GETT_FLOAT32) {
                    const float a = (float)alpha, b = (float)be;
                    return rocblas_sgemm_strided_batched(
                        h, ta, tb, m, n, k, &a, (const float *)(L + oL), lda, bL,
                        (const float *)(R + oR), ldb, bR, &b, (float *)(Cb + oC), ldc, bC, batch);
                }
                return rocblas_dgemm_strided_batched(
                    h, ta, tb, m, n, k, &alpha, (const double *)(L + oL), lda, bL,
                    (const double *)(R + oR), ldb, bR, &be, (double *)(Cb + oC), ldc, bC, batch);
            });
            if (st != GETT_SUCCESS) return st;
            size_t i = 0;
            for (; i < qf.size(); ++i) {
                const gett::LoopIdx &l = P.freeLoops[i];
                fOffL += l.sL;
                fOffR += l.sR;
                fOffC += l.sC;
                if (++qf[i] < l.extent) break;
                fOffL -= l.sL * l.extent;
                fOffR -= l.sR * l.extent;
                fOffC -= l.sC * l.extent;
                qf[i] = 0;
            }
            if (i == qf.size()) break;
        }
        size_t j = 0;
        for (; j < qk.size(); ++j) {
            const gett::LoopIdx &l = P.kLoops[j];
            kOffL += l.sL;
            kOffR += l.sR;
            if (++qk[j] < l.extent) break;
            kOffL -= l.sL * l.extent;
            kOffR -= l.sR * l.extent;
            qk[j] = 0;
        }
        if (j == qk.size()) break;
    }
    return GETT_SUCCESS;
}

gett_status_t gett_log_destroy(gett_log_plan_t plan)
{
    delete plan;
    return GETT_SUCCESS;
}

const char *gett_log_describe(const gett_log_plan_t plan)
{
    return plan ? plan->text.c_str() : "";
}

}  // extern "C"
