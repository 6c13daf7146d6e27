// ttgt.cpp -- Transpose-Transpose-GEMM-Transpose (Sec. 4), the method GETT is
// measured against, and the stand-alone transposition of Eq. 4.
//
// TTGT flattens the operands into matrices with explicit transpositions,
// multiplies them with a library GEMM and folds the product back into C.
// Planning follows Sec. 4: for orders of I_m, I_n and I_k, eight operand
// arrangements (which operand is the GEMM's left one, and whether each is
// stored free-index-major or contracted-index-major) are costed by the number
// of elements that must be transposed; ties go to the candidate whose
// transpositions keep each tensor's stride-one index.  A tensor whose layout
// already is the required matrix (unit-stride rows, one leading dimension) is
// used in place.
//
// Orders considered for each set: the order in which each of the two tensors
// holding it stores it.  Any other order forces both of those tensors to be
// transposed, so it never costs fewer elements than one of these.
//
// The GEMM is rocBLAS (column-major sgemm / dgemm); the transpositions and the
// fold are this library's Eq. 4 kernel.  Workspace is provided by the caller.
#include <hip/hip_runtime_api.h>
#include <rocblas/rocblas.h>
#include <stdint.h>
#include <string.h>

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

constexpr int64_t kAlign = 256;   // workspace regions start on 256-byte boundaries

int64_t stride_in(const Index &x, int t) { return t == 0 ? x.strC : t == 1 ? x.strA : x.strB; }

int64_t size_of(const std::vector<Index> &s)
{
    int64_t n = 1;
    for (auto &x : s) n *= x.extent;
    return n;
}

// Leading dimension of the column-major matrix (rows, cols) when tensor t is
// already laid out as that matrix, else -1.
int64_t matrix_ld(const std::vector<Index> &rows, const std::vector<Index> &cols, int t)
{
    int64_t next = 1;
    for (auto &x : rows) {
        if (stride_in(x, t) != next) return -1;
        next *= x.extent;
    }
    const int64_t nrows = next;
    if (cols.empty()) return nrows;
    const int64_t ld = stride_in(cols[0], t);
    if (ld < nrows) return -1;
    next = ld;
    for (auto &x : cols) {
        if (stride_in(x, t) != next) return -1;
        next *= x.extent;
    }
    return ld;
}

// One explicit transposition: iteration space with source and target strides.
struct Move {
    bool active = false;
    std::vector<int64_t> ext, src, dst;
    int64_t offset = 0;   // workspace byte offset of the matrix (operands and X)
};

// The matrix (rows, cols) of tensor t, dense in the workspace.
Move to_matrix(const std::vector<Index> &rows, const std::vector<Index> &cols, int t)
{
    Move m;
    m.active = true;
    int64_t acc = 1;
    for (const auto *g : {&rows, &cols})
        for (auto &x : *g) {
            m.ext.push_back(x.extent);
            m.src.push_back(stride_in(x, t));
            m.dst.push_back(acc);
            acc *= x.extent;
        }
    return m;
}

struct GemmOperand {
    int tensor = 1;                 // 1: A, 2: B
    bool opT = false;               // stored contracted-index-major
    int64_t ld = 1;
    Move move;                      // active when the operand is transposed first
};

struct Flattening {
    std::vector<Index> Pm, Pn, Pk;
    bool leftA = true;
    bool leftFreeFirst = true, rightKFirst = true;
    int64_t cost = 0, workspace = 0;
    int changes = 0;
    GemmOperand L, R;
    bool fold = false;
    int64_t ldX = 1;
    Move foldMove;
};

std::string names(const std::vector<Index> &s)
{
    std::string o;
    for (size_t i = 0; i < s.size(); ++i) o += (i ? "," : "") + s[i].name;
    return o;
}

// Name of tensor t's stride-one (smallest-stride) index among the given sets.
std::string unit_index(const std::vector<const std::vector<Index> *> &sets, int t)
{
    int64_t best = INT64_MAX;
    std::string n;
    for (auto *s : sets)
        for (auto &x : *s)
            if (stride_in(x, t) < best) {
                best = stride_in(x, t);
                n = x.name;
            }
    return n;
}

std::vector<std::vector<Index>> orders(const std::vector<Index> &s, int t1, int t2)
{
    std::vector<std::vector<Index>> out;
    for (int t : {t1, t2}) {
        std::vector<Index> o = s;
        std::stable_sort(o.begin(), o.end(),
                         [t](const Index &a, const Index &b) { return stride_in(a, t) < stride_in(b, t); });
        bool dup = false;
        for (auto &p : out) dup |= names(p) == names(o);
        if (!dup) out.push_back(o);
    }
    return out;
}

}  // namespace
}  // namespace gett

struct gett_ttgt_plan_s {
    gett_dtype_t dtype;
    gett::Analysis an;
    gett::Flattening best;
    int64_t M = 1, N = 1, K = 1;
    int64_t workspace = 0;
    int considered = 0;
    std::vector<int64_t> cExt, cStr;   // C's iteration space (for C <- beta * C)
    std::string text;
};

namespace gett {
namespace {

gett_status_t plan_ttgt(gett_ttgt_plan_s &P, int64_t maxWorkspace)
{
    const Analysis &an = P.an;
    const int64_t item = P.dtype == GETT_FLOAT32 ? 4 : 8;
    const int64_t sizeA = an.sizeM * an.sizeK, sizeB = an.sizeN * an.sizeK,
                  sizeC = an.sizeM * an.sizeN;
    auto pad = [](int64_t b) { return (b + kAlign - 1) / kAlign * kAlign; };
    bool found = false;
    for (auto &pm : orders(an.Im, 1, 0))
        for (auto &pn : orders(an.In, 2, 0))
            for (auto &pk : orders(an.Ik, 1, 2))
                for (int arr = 0; arr < 8; ++arr) {
                    Flattening c;
                    c.Pm = pm;
                    c.Pn = pn;
                    c.Pk = pk;
                    c.leftA = !(arr & 4);
                    c.leftFreeFirst = !(arr & 2);
                    c.rightKFirst = !(arr & 1);
                    const std::vector<Index> &FL = c.leftA ? pm : pn, &FR = c.leftA ? pn : pm;
                    c.L.tensor = c.leftA ? 1 : 2;
                    c.R.tensor = c.leftA ? 2 : 1;
                    c.L.opT = !c.leftFreeFirst;
                    c.R.opT = !c.rightKFirst;
                    const std::vector<Index> &lr = c.leftFreeFirst ? FL : pk, &lc = c.leftFreeFirst ? pk : FL;
                    const std::vector<Index> &rr = c.rightKFirst ? pk : FR, &rc = c.rightKFirst ? FR : pk;
                    const std::vector<const std::vector<Index> *> setsL = {&FL, &pk}, setsR = {&FR, &pk},
                                                                  setsC = {&FL, &FR};
                    int64_t ws = 0;
                    auto place = [&](GemmOperand &o, const std::vector<Index> &rows,
                                     const std::vector<Index> &cols,
                                     const std::vector<const std::vector<Index> *> &sets) {
                        o.ld = matrix_ld(rows, cols, o.tensor);
                        if (o.ld >= 0) return;
                        o.move = to_matrix(rows, cols, o.tensor);
                        o.move.offset = ws;
                        o.ld = std::max<int64_t>(size_of(rows), 1);
                        const int64_t n = size_of(rows) * size_of(cols);
                        ws += pad(n * item);
                        c.cost += n;
                        const std::string newUnit = rows.empty() ? (cols.empty() ? "" : cols[0].name)
                                                                 : rows[0].name;
                        c.changes += unit_index(sets, o.tensor) != newUnit;
                    };
                    place(c.L, lr, lc, setsL);
                    place(c.R, rr, rc, setsR);
                    c.ldX = matrix_ld(FL, FR, 0);
                    if (c.ldX < 0) {
                        c.fold = true;
                        c.ldX = std::max<int64_t>(size_of(FL), 1);
                        // X (dense, FL x FR) -> C
                        Move f;
                        f.active = true;
                        f.offset = ws;
                        int64_t acc = 1;
                        for (const auto *g : {&FL, &FR})
                            for (auto &x : *g) {
                                f.ext.push_back(x.extent);
                                f.src.push_back(acc);
                                f.dst.push_back(x.strC);
                                acc *= x.extent;
                            }
                        c.foldMove = f;
                        ws += pad(sizeC * item);
                        c.cost += sizeC;
                        c.changes += unit_index(setsC, 0) != (FL.empty() ? (FR.empty() ? "" : FR[0].name)
                                                                          : FL[0].name);
                    }
                    c.workspace = ws;
                    ++P.considered;
                    if (maxWorkspace >= 0 && ws > maxWorkspace) continue;
                    const Flattening &b = P.best;
                    if (!found || c.cost < b.cost || (c.cost == b.cost && c.changes < b.changes) ||
                        (c.cost == b.cost && c.changes == b.changes && c.workspace < b.workspace)) {
                        P.best = c;
                        found = true;
                    }
                }
    (void)sizeA;
    (void)sizeB;
    if (!found) return GETT_ERROR_NOT_SUPPORTED;
    const Flattening &b = P.best;
    P.M = std::max<int64_t>(size_of(b.leftA ? b.Pm : b.Pn), 1);
    P.N = std::max<int64_t>(size_of(b.leftA ? b.Pn : b.Pm), 1);
    P.K = std::max<int64_t>(size_of(b.Pk), 1);
    P.workspace = b.workspace;
    for (int64_t v : {P.M, P.N, P.K, b.L.ld, b.R.ld, b.ldX})
        if (v > INT32_MAX) return GETT_ERROR_NOT_SUPPORTED;
    return GETT_SUCCESS;
}

void describe(gett_ttgt_plan_s &P)
{
    const Flattening &b = P.best;
    const char *tn[3] = {"C", "A", "B"};
    std::ostringstream o;
    o << "{\"method\":\"ttgt\",\"dtype\":\"" << (P.dtype == GETT_FLOAT32 ? "f32" : "f64") << "\"";
    o << ",\"order_m\":\"" << names(b.Pm) << "\",\"order_n\":\"" << names(b.Pn) << "\",\"order_k\":\""
      << names(b.Pk) << "\"";
    o << ",\"gemm\":{\"left\":\"" << tn[b.L.tensor] << "\",\"right\":\"" << tn[b.R.tensor]
      << "\",\"op_left\":\"" << (b.L.opT ? "T" : "N") << "\",\"op_right\":\"" << (b.R.opT ? "T" : "N")
      << "\",\"m\":" << P.M << ",\"n\":" << P.N << ",\"k\":" << P.K << ",\"lda\":" << b.L.ld
      << ",\"ldb\":" << b.R.ld << ",\"ldc\":" << b.ldX << "}";
    o << ",\"transposed\":[";
    bool first = true;
    for (const GemmOperand *op : {&b.L, &b.R})
        if (op->move.active) {
            o << (first ? "" : ",") << "\"" << tn[op->tensor] << "\"";
            first = false;
        }
    if (b.fold) o << (first ? "" : ",") << "\"C\"";
    o << "],\"transposed_elements\":" << b.cost << ",\"stride_one_changes\":" << b.changes
      << ",\"workspace_bytes\":" << P.workspace << ",\"candidates\":" << P.considered
      << ",\"empty_c\":" << (P.an.emptyC ? "true" : "false")
      << ",\"empty_sum\":" << (P.an.emptySum ? "true" : "false") << "}";
    P.text = o.str();
}

gett_status_t gemm(const gett_ttgt_plan_s &P, double alpha, const void *L, const void *R,
                   double beta, void *X, hipStream_t stream)
{
    const Flattening &b = P.best;
    const rocblas_operation ta = b.L.opT ? rocblas_operation_transpose : rocblas_operation_none;
    const rocblas_operation tb = b.R.opT ? rocblas_operation_transpose : rocblas_operation_none;
    const rocblas_int m = (rocblas_int)P.M, n = (rocblas_int)P.N, k = (rocblas_int)P.K;
    const rocblas_int lda = (rocblas_int)b.L.ld, ldb = (rocblas_int)b.R.ld, ldc = (rocblas_int)b.ldX;
    return with_blas(stream, [&](rocblas_handle h) {
        if (P.dtype == GETT_FLOAT32) {
            const float a = (float)alpha, c = (float)beta;
            return rocblas_sgemm(h, ta, tb, m, n, k, &a, (const float *)L, lda, (const float *)R,
                                 ldb, &c, (float *)X, ldc);
        }
        return rocblas_dgemm(h, ta, tb, m, n, k, &alpha, (const double *)L, lda,
                             (const double *)R, ldb, &beta, (double *)X, ldc);
    });
}

gett_status_t run_move(const gett_ttgt_plan_s &P, const Move &m, double alpha, const void *src,
                       double beta, void *dst, hipStream_t stream)
{
    return transpose_launch(P.dtype, (int)m.ext.size(), m.ext.data(), m.src.data(), m.dst.data(),
                            alpha, src, beta, dst, stream);
}

int64_t max_off(int rank, const int64_t *ext, const int64_t *str)
{
    int64_t m = 0;
    for (int i = 0; i < rank; ++i) {
        if (ext[i] <= 1) continue;
        if (str[i] >= INT32_MAX) return INT64_MAX;
        m += (ext[i] - 1) * str[i];
        if (m >= INT32_MAX) return INT64_MAX;
    }
    return m;
}

}  // namespace
}  // namespace gett

extern "C" {

gett_status_t gett_transpose(gett_dtype_t dtype, int rank, const int64_t *extent,
                             const int64_t *stride_in, const int64_t *stride_out, double alpha,
                             const void *in, double beta, void *out, void *stream)
{
    if (dtype != GETT_FLOAT32 && dtype != GETT_FLOAT64) return GETT_ERROR_INVALID_VALUE;
    if (rank < 0) return GETT_ERROR_INVALID_VALUE;
    if (rank > GETT_MAX_RANK) return GETT_ERROR_NOT_SUPPORTED;
    if (rank > 0 && !extent) return GETT_ERROR_INVALID_VALUE;
    int64_t ext[GETT_MAX_RANK], si[GETT_MAX_RANK], so[GETT_MAX_RANK];
    int64_t accI = 1, accO = 1;
    bool empty = false;
    for (int i = 0; i < rank; ++i) {
        ext[i] = extent[i];
        if (ext[i] < 0 || ext[i] > INT32_MAX) return GETT_ERROR_INVALID_VALUE;
        empty |= ext[i] == 0;
        si[i] = stride_in ? stride_in[i] : accI;
        so[i] = stride_out ? stride_out[i] : accO;
        accI *= std::max<int64_t>(ext[i], 1);
        accO *= std::max<int64_t>(ext[i], 1);
        if (si[i] < 0 || so[i] < 0) return GETT_ERROR_INVALID_VALUE;
        if (ext[i] > 1 && (si[i] < 1 || so[i] < 1)) return GETT_ERROR_INVALID_VALUE;
    }
    const int64_t item = dtype == GETT_FLOAT32 ? 4 : 8;
    if (!out || (uintptr_t)out % item) return GETT_ERROR_INVALID_VALUE;
    const bool readIn = alpha != 0.0;
    if (readIn && (!in || (uintptr_t)in % item)) return GETT_ERROR_INVALID_VALUE;
    if (empty) return GETT_SUCCESS;
    const int64_t mi = gett::max_off(rank, ext, si), mo = gett::max_off(rank, ext, so);
    if (mi >= INT32_MAX || mo >= INT32_MAX) return GETT_ERROR_NOT_SUPPORTED;
    if (!gett::strides_injective(rank, ext, so)) return GETT_ERROR_NOT_SUPPORTED;
    if (readIn && gett::overlaps(in, (mi + 1) * item, out, (mo + 1) * item))
        return GETT_ERROR_INVALID_VALUE;
    return gett::transpose_launch(dtype, rank, ext, si, so, alpha, in, beta, out,
                                  (hipStream_t)stream);
}

gett_status_t gett_ttgt_plan(gett_ttgt_plan_t *plan, gett_dtype_t dtype, const char *modes_C,
                             const int64_t *extent_C, const int64_t *stride_C, const char *modes_A,
                             const int64_t *extent_A, const int64_t *stride_A, const char *modes_B,
                             const int64_t *extent_B, const int64_t *stride_B,
                             int64_t max_workspace_bytes)
{
    if (!plan) return GETT_ERROR_INVALID_VALUE;
    *plan = nullptr;
    gett_ttgt_plan_s *p = new (std::nothrow) gett_ttgt_plan_s();
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
            if (!p->an.emptyC && !p->an.emptySum) st = gett::plan_ttgt(*p, max_workspace_bytes);
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

gett_status_t gett_ttgt_workspace_size(const gett_ttgt_plan_t plan, uint64_t *bytes)
{
    if (!plan || !bytes) return GETT_ERROR_INVALID_VALUE;
    *bytes = (uint64_t)plan->workspace;
    return GETT_SUCCESS;
}

gett_status_t gett_ttgt_contract(const gett_ttgt_plan_t plan, double alpha, const void *A,
                                 const void *B, double beta, void *C, void *workspace,
                                 uint64_t workspace_bytes, void *stream)
{
    if (!plan) return GETT_ERROR_INVALID_VALUE;
    const gett_ttgt_plan_s &P = *plan;
    if (P.an.emptyC) return GETT_SUCCESS;
    const bool readAB = alpha != 0.0 && !P.an.emptySum;
    if (!gett::operands_ok(P.dtype, P.an, readAB, A, B, C)) return GETT_ERROR_INVALID_VALUE;
    hipStream_t s = (hipStream_t)stream;
    if (!readAB)   // C <- beta * C
        return gett::transpose_launch(P.dtype, (int)P.cExt.size(), P.cExt.data(), P.cStr.data(),
                                      P.cStr.data(), 0.0, nullptr, beta, C, s);
    const gett::Flattening &b = P.best;
    if (P.workspace > 0) {
        if (!workspace || workspace_bytes < (uint64_t)P.workspace ||
            (uintptr_t)workspace % gett::kAlign)
            return GETT_ERROR_INVALID_VALUE;
        const int64_t item = P.dtype == GETT_FLOAT32 ? 4 : 8;
        if (gett::overlaps(workspace, P.workspace, C, (P.an.maxOffC + 1) * item) ||
            gett::overlaps(workspace, P.workspace, A, (P.an.maxOffA + 1) * item) ||
            gett::overlaps(workspace, P.workspace, B, (P.an.maxOffB + 1) * item))
            return GETT_ERROR_INVALID_VALUE;
    }
    char *ws = static_cast<char *>(workspace);
    const void *src[3] = {C, A, B};
    const void *ops[2];
    const gett::GemmOperand *o2[2] = {&b.L, &b.R};
    gett_status_t st;
    for (int i = 0; i < 2; ++i) {
        const gett::GemmOperand &o = *o2[i];
        if (o.move.active) {
            void *dst = ws + o.move.offset;
            st = gett::run_move(P, o.move, 1.0, src[o.tensor], 0.0, dst, s);
            if (st != GETT_SUCCESS) return st;
            ops[i] = dst;
        } else {
            ops[i] = src[o.tensor];
        }
    }
    void *X = b.fold ? static_cast<void *>(ws + b.foldMove.offset) : C;
    st = gett::gemm(P, alpha, ops[0], ops[1], b.fold ? 0.0 : beta, X, s);
    if (st != GETT_SUCCESS) return st;
    if (b.fold) return gett::run_move(P, b.foldMove, 1.0, X, beta, C, s);
    return GETT_SUCCESS;
}

gett_status_t gett_ttgt_destroy(gett_ttgt_plan_t plan)
{
    delete plan;
    return GETT_SUCCESS;
}

const char *gett_ttgt_describe(const gett_ttgt_plan_t plan)
{
    return plan ? plan->text.c_str() : "";
}

}  // extern "C"
