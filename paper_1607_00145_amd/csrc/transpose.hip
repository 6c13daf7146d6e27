// transpose.hip -- general tensor transposition with input and output
// scaling (Sec. 2.3, Eq. 4):
//
//     out[Pi(i)] <- alpha * in[i] + beta * out[Pi(i)]
//
// The permutation is carried by the strides: index d of the iteration space
// has stride sin[d] in the input and sout[d] in the output.
//
// Design (HBM-bound; one read of the input, one write of the output, plus a
// read of the output when beta != 0):
//   * indices are split into three groups: P, the input's fastest indices
//     (their product reaches the tile edge), Q, the output's fastest
//     indices among the rest, and R, everything else;
//   * one workgroup moves a TE x TE tile of the (P, Q) plane for one point of
//     R.  Reads run along P (contiguous in the input), the tile passes
//     through LDS, and writes run along Q (contiguous in the output) -- or
//     along P when the output's stride-one index is itself in P;
//   * the element offsets of the tile's P and Q positions are decoded once
//     per workgroup into small LDS tables, so the copy loops do no index
//     arithmetic beyond two table reads.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <vector>

#include "transpose.hpp"

namespace gett {
namespace {

constexpr int kTE = 64;        // tile edge (elements)
constexpr int kThreads = 256;  // 4 waves
constexpr int kRows = kThreads / kTE;

struct TDesc {
    int32_t n[3];                    // indices in P, Q, R
    int32_t ext[3][kMaxDims];
    int32_t sin[3][kMaxDims];
    int32_t sout[3][kMaxDims];
    int32_t size[3];                 // products of the extents of P, Q, R
    int32_t tiles[2];                // tiles along P and Q
    int32_t alongP;                  // the output's stride-one index is in P
};

// Offsets of the linear position `lin` of group g in the input and output.
__device__ inline void decode(const TDesc &d, int g, int32_t lin, int32_t &oi, int32_t &oo)
{
    oi = 0;
    oo = 0;
    for (int i = 0; i < d.n[g]; ++i) {
        const int32_t e = d.ext[g][i];
        const int32_t x = lin % e;
        lin /= e;
        oi += x * d.sin[g][i];
        oo += x * d.sout[g][i];
    }
}

template <typename T>
__global__ __launch_bounds__(kThreads) void transpose_kernel(const TDesc d, const T *__restrict__ in,
                                                             T *__restrict__ out, T alpha, T beta)
{
    __shared__ T tile[kTE][kTE + 1];   // [q][p]
    __shared__ int32_t pin[kTE], pout[kTE], qin[kTE], qout[kTE];

    const uint32_t b = blockIdx.x;
    const int32_t tp = (int32_t)(b % (uint32_t)d.tiles[0]);
    const uint32_t rest = b / (uint32_t)d.tiles[0];
    const int32_t tq = (int32_t)(rest % (uint32_t)d.tiles[1]);
    const int32_t r = (int32_t)(rest / (uint32_t)d.tiles[1]);
    int32_t rin, rout;
    decode(d, 2, r, rin, rout);

    const int t = threadIdx.x;
    if (t < kTE) {
        const int32_t p = tp * kTE + t;
        int32_t oi = -1, oo = -1;
        if (p < d.size[0]) decode(d, 0, p, oi, oo);
        pin[t] = oi;
        pout[t] = oo;
    } else if (t < 2 * kTE) {
        const int32_t q = tq * kTE + (t - kTE);
        int32_t oi = -1, oo = -1;
        if (q < d.size[1]) decode(d, 1, q, oi, oo);
        qin[t - kTE] = oi;
        qout[t - kTE] = oo;
    }
    __syncthreads();

    const T *src = in + rin;
    T *dst = out + rout;
    const int lane = t % kTE, row = t / kTE;
    const bool readIn = alpha != T(0);
    // read along P: lanes take consecutive P positions
    if (readIn) {
        const int32_t oi = pin[lane];
#pragma unroll
        for (int j = 0; j < kTE / kRows; ++j) {
            const int ql = row + kRows * j;
            const int32_t qo = qin[ql];
            T v = T(0);
            if (oi >= 0 && qo >= 0) v = src[oi + qo];
            tile[ql][lane] = v;
        }
    }
    __syncthreads();
    if (d.alongP) {   // write along P
        const int32_t oo = pout[lane];
        if (oo < 0) return;
#pragma unroll
        for (int j = 0; j < kTE / kRows; ++j) {
            const int ql = row + kRows * j;
            const int32_t qo = qout[ql];
            if (qo < 0) continue;
            T v = readIn ? alpha * tile[ql][lane] : T(0);
            if (beta != T(0)) v = beta * dst[oo + qo] + v;
            dst[oo + qo] = v;
        }
    } else {          // write along Q: lanes take consecutive Q positions
        const int32_t qo = qout[lane];
        if (qo < 0) return;
#pragma unroll
        for (int j = 0; j < kTE / kRows; ++j) {
            const int pl = row + kRows * j;
            const int32_t oo = pout[pl];
            if (oo < 0) continue;
            T v = readIn ? alpha * tile[lane][pl] : T(0);
            if (beta != T(0)) v = beta * dst[oo + qo] + v;
            dst[oo + qo] = v;
        }
    }
}

struct Idx {
    int64_t ext, sin, sout;
};

}  // namespace

gett_status_t transpose_launch(gett_dtype_t dtype, int rank, const int64_t *ext,
                               const int64_t *sin, const int64_t *sout, double alpha,
                               const void *in, double beta, void *out, hipStream_t stream)
{
    // drop extent-1 indices; an empty extent means nothing to do
    std::vector<Idx> v;
    for (int i = 0; i < rank; ++i) {
        if (ext[i] == 0) return GETT_SUCCESS;
        if (ext[i] > 1) v.push_back({ext[i], sin[i], sout[i]});
    }
    // merge an index into another when it follows it in both layouts
    for (bool changed = true; changed;) {
        changed = false;
        for (size_t p = 0; p < v.size() && !changed; ++p)
            for (size_t q = 0; q < v.size() && !changed; ++q) {
                if (p == q) continue;
                if (v[q].sin == v[p].sin * v[p].ext && v[q].sout == v[p].sout * v[p].ext) {
                    v[p].ext *= v[q].ext;
                    v.erase(v.begin() + q);
                    changed = true;
                }
            }
    }
    // P: by input stride until the tile edge is covered; Q: by output stride
    std::vector<Idx> byIn = v, P, Q, R;
    std::stable_sort(byIn.begin(), byIn.end(), [](const Idx &a, const Idx &b) { return a.sin < b.sin; });
    int64_t sp = 1, sq = 1;
    size_t i = 0;
    for (; i < byIn.size() && sp < kTE; ++i) {
        P.push_back(byIn[i]);
        sp *= byIn[i].ext;
    }
    std::vector<Idx> others(byIn.begin() + i, byIn.end());
    std::stable_sort(others.begin(), others.end(), [](const Idx &a, const Idx &b) { return a.sout < b.sout; });
    size_t j = 0;
    for (; j < others.size() && sq < kTE; ++j) {
        Q.push_back(others[j]);
        sq *= others[j].ext;
    }
    R.assign(others.begin() + j, others.end());
    if (Q.empty() && P.size() > 1) {   // give the Q side an index of its own
        Q.push_back(P.back());
        sq = P.back().ext;
        sp /= P.back().ext;
        P.pop_back();
    }
    int64_t sr = 1;
    for (auto &x : R) sr *= x.ext;
    if (sp >= INT32_MAX || sq >= INT32_MAX || sr >= INT32_MAX) return GETT_ERROR_NOT_SUPPORTED;

    TDesc d = {};
    const std::vector<Idx> *groups[3] = {&P, &Q, &R};
    for (int g = 0; g < 3; ++g) {
        d.n[g] = (int32_t)groups[g]->size();
        for (int k = 0; k < d.n[g]; ++k) {
            const Idx &x = (*groups[g])[k];
            d.ext[g][k] = (int32_t)x.ext;
            d.sin[g][k] = (int32_t)x.sin;
            d.sout[g][k] = (int32_t)x.sout;
        }
    }
    d.size[0] = (int32_t)sp;
    d.size[1] = (int32_t)sq;
    d.size[2] = (int32_t)sr;
    d.tiles[0] = (int32_t)((sp + kTE - 1) / kTE);
    d.tiles[1] = (int32_t)((sq + kTE - 1) / kTE);
    // the output's smallest stride decides the write direction
    int64_t minOut = INT64_MAX;
    bool inP = true;
    for (auto &x : P)
        if (x.sout < minOut) { minOut = x.sout; inP = true; }
    for (auto &x : Q)
        if (x.sout < minOut) { minOut = x.sout; inP = false; }
    for (auto &x : R)
        if (x.sout < minOut) { minOut = x.sout; inP = false; }
    d.alongP = inP ? 1 : 0;
    const int64_t blocks = (int64_t)d.tiles[0] * d.tiles[1] * sr;
    if (blocks >= INT32_MAX) return GETT_ERROR_NOT_SUPPORTED;
    if (blocks == 0) return GETT_SUCCESS;
    if (dtype == GETT_FLOAT32)
        hipLaunchKernelGGL(transpose_kernel<float>, dim3((unsigned)blocks), dim3(kThreads), 0, stream,
                           d, static_cast<const float *>(in), static_cast<float *>(out),
                           (float)alpha, (float)beta);
    else
        hipLaunchKernelGGL(transpose_kernel<double>, dim3((unsigned)blocks), dim3(kThreads), 0,
                           stream, d, static_cast<const double *>(in), static_cast<double *>(out),
                           alpha, beta);
    return hipGetLastError() == hipSuccess ? GETT_SUCCESS : GETT_ERROR_HIP;
}

}  // namespace gett
