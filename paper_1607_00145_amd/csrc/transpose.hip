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
//   * one workgroup moves a TP x TQ tile of the (P, Q) plane for one point of
//     R.  Reads run along P (contiguous in the input), the tile passes
//     through LDS, and writes run along Q (contiguous in the output) -- or
//     along P when the output's stride-one index is itself in P;
//   * the element offsets of the tile's P and Q positions are decoded once
//     per workgroup into small LDS tables, so the copy loops do no index
//     arithmetic beyond two table reads.
#include <hip/hip_runtime.h>

#include <stdint.h>

#include <algorithm>
#include <atomic>
#include <type_traits>
#include <vector>

#include "transpose.hpp"

namespace gett {
namespace {

// Tile edges along P and Q (elements) and threads per workgroup.
template <typename T> struct Shape;
template <> struct Shape<float> { static constexpr int TP = 128, TQ = 128, TH = 512; };
template <> struct Shape<double> { static constexpr int TP = 64, TQ = 64, TH = 256; };

struct TDesc {
    int32_t n[3];                    // indices in P, Q, R
    int32_t ext[3][kMaxDims];
    int32_t sin[3][kMaxDims];
    int32_t sout[3][kMaxDims];
    int32_t size[3];                 // products of the extents of P, Q, R
    int32_t tiles[2];                // tiles along P and Q
    int32_t alongP;                  // the output's stride-one index is in P
    int32_t group;                   // > 0: walk tiles in bands of this many P tiles
};

// Tile (tp, tq) and point r of R moved by workgroup b.  Tiles run P-fastest:
// the workgroups resident at one time read neighbouring stretches of the
// same input rows and, when they span several Q tiles, write neighbouring
// stretches of the same output rows.  When one row of P tiles alone fills
// the device, bands of `group` P tiles keep several Q tiles in flight, or
// every write run of 16-byte vectors would stand alone in its DRAM page.
__device__ inline void tile_of(const TDesc &d, uint32_t b, int32_t &tp, int32_t &tq, int32_t &r)
{
    const uint32_t t0 = (uint32_t)d.tiles[0], t1 = (uint32_t)d.tiles[1];
    const uint32_t per = t0 * t1;
    r = (int32_t)(b / per);
    const uint32_t t = b - (uint32_t)r * per;
    if (d.group <= 0) {
        tp = (int32_t)(t % t0);
        tq = (int32_t)(t / t0);
        return;
    }
    const uint32_t g = (uint32_t)d.group, band = g * t1;
    const uint32_t first = (t / band) * g;
    const uint32_t gsz = min(t0 - first, g);
    const uint32_t in = t - (t / band) * band;
    tp = (int32_t)(first + in % gsz);
    tq = (int32_t)(in / gsz);
}

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

template <typename T> struct Vec;
template <> struct Vec<float> { typedef float __attribute__((ext_vector_type(4))) type; static constexpr int n = 4; };
template <> struct Vec<double> { typedef double __attribute__((ext_vector_type(2))) type; static constexpr int n = 2; };

// The phases of moving one tile.  VL / VS: 16-byte vector reads along P /
// writes along the output's stride-one side (the host has checked that every
// vector lies within one index run and is aligned); ALONGP: the output's
// stride-one index is in P.
template <typename T, bool VL, bool VS, bool ALONGP>
struct Mover {
    static constexpr int kTP = Shape<T>::TP, kTQ = Shape<T>::TQ, kThreads = Shape<T>::TH;
    typedef typename Vec<T>::type vec;
    static constexpr int VW = Vec<T>::n;
    static constexpr int RL = VL ? VW : 1;   // elements per read
    static constexpr int RS = VS ? VW : 1;   // elements per write
    static constexpr int PERL = kTP / RL;    // reading threads per Q row
    static constexpr int NL = kTQ * PERL / kThreads;
    static_assert(kTP + kTQ <= kThreads, "one table entry per thread");

    // offset tables of tile b (-1: outside the tensor) and its R offsets
    static __device__ __forceinline__ void tables(const TDesc &d, uint32_t b, int t,
                                                  int32_t *pin, int32_t *pout, int32_t *qin,
                                                  int32_t *qout, int32_t &rin, int32_t &rout)
    {
        int32_t tp, tq, r;
        tile_of(d, b, tp, tq, r);
        decode(d, 2, r, rin, rout);
        if (t < kTP) {
            const int32_t p = tp * kTP + t;
            int32_t oi = -1, oo = -1;
            if (p < d.size[0]) decode(d, 0, p, oi, oo);
            pin[t] = oi;
            pout[t] = oo;
        } else if (t < kTP + kTQ) {
            const int32_t q = tq * kTQ + (t - kTP);
            int32_t oi = -1, oo = -1;
            if (q < d.size[1]) decode(d, 1, q, oi, oo);
            qin[t - kTP] = oi;
            qout[t - kTP] = oo;
        }
    }

    // read along P: a thread takes RL consecutive P positions of NL Q rows
    static __device__ __forceinline__ void load(const T *src, const int32_t *pin,
                                                const int32_t *qin, int t, T (&v)[NL][RL])
    {
        const int pl = (t % PERL) * RL;
        const int32_t oi = pin[pl];
        int32_t qo[NL];   // every table read first: one LDS wait, then the loads
#pragma unroll
        for (int j = 0; j < NL; ++j) qo[j] = qin[t / PERL + (kThreads / PERL) * j];
#pragma unroll
        for (int j = 0; j < NL; ++j) {
            if (oi >= 0 && qo[j] >= 0) {
                if constexpr (VL) {
                    const vec x = *reinterpret_cast<const vec *>(src + oi + qo[j]);
#pragma unroll
                    for (int e = 0; e < RL; ++e) v[j][e] = x[e];
                } else {
                    v[j][0] = src[oi + qo[j]];
                }
            } else {
#pragma unroll
                for (int e = 0; e < RL; ++e) v[j][e] = T(0);
            }
        }
    }

    static __device__ __forceinline__ void stash(T (*tile)[kTP + 1], int t, const T (&v)[NL][RL])
    {
        const int pl = (t % PERL) * RL;
#pragma unroll
        for (int j = 0; j < NL; ++j) {
            const int ql = t / PERL + (kThreads / PERL) * j;
#pragma unroll
            for (int e = 0; e < RL; ++e) tile[ql][pl + e] = v[j][e];
        }
    }

    // write: a thread takes RS consecutive positions along the output's
    // stride-one side (P when ALONGP, else Q)
    static __device__ __forceinline__ void write(T *dst, const int32_t *pout, const int32_t *qout,
                                                 const T (*tile)[kTP + 1], int t, T alpha, T beta,
                                                 bool readIn, bool readOut)
    {
        constexpr int LEN = ALONGP ? kTP : kTQ;   // tile edge along the write direction
        constexpr int PER = LEN / RS;
        constexpr int N = (kTP * kTQ / LEN) * PER / kThreads;
        const int a = (t % PER) * RS;   // position along the write direction
        int32_t off[N];                   // output offsets, -1 outside the tensor
#pragma unroll
        for (int j = 0; j < N; ++j) {
            const int c = t / PER + (kThreads / PER) * j;   // position across it
            const int pl = ALONGP ? a : c, ql = ALONGP ? c : a;
            const int32_t oo = pout[pl], qo = qout[ql];
            off[j] = oo < 0 || qo < 0 ? -1 : oo + qo;
        }
#pragma unroll
        for (int j = 0; j < N; ++j) {
            const int c = t / PER + (kThreads / PER) * j;
            const int pl = ALONGP ? a : c, ql = ALONGP ? c : a;
            if (off[j] < 0) continue;
            T *o = dst + off[j];
            T w[RS];
#pragma unroll
            for (int e = 0; e < RS; ++e)
                w[e] = readIn ? alpha * (ALONGP ? tile[ql][pl + e] : tile[ql + e][pl]) : T(0);
            if constexpr (VS) {
                vec x;
                if (readOut) {
                    const vec old = *reinterpret_cast<const vec *>(o);
#pragma unroll
                    for (int e = 0; e < RS; ++e) x[e] = beta * old[e] + w[e];
                } else {
#pragma unroll
                    for (int e = 0; e < RS; ++e) x[e] = w[e];
                }
                *reinterpret_cast<vec *>(o) = x;
            } else {
                *o = readOut ? beta * *o + w[0] : w[0];
            }
        }
    }
};

// One tile per workgroup: tables, read into LDS, write out.
template <typename T, bool VL, bool VS, bool ALONGP>
__global__ __launch_bounds__(Shape<T>::TH) void transpose_kernel(const TDesc d, const T *__restrict__ in,
                                                                 T *__restrict__ out, T alpha, T beta)
{
    typedef Mover<T, VL, VS, ALONGP> M;
    __shared__ T tile[M::kTQ][M::kTP + 1];   // [q][p]
    __shared__ int32_t pin[M::kTP], pout[M::kTP], qin[M::kTQ], qout[M::kTQ];
    const int t = threadIdx.x;
    int32_t rin, rout;
    M::tables(d, blockIdx.x, t, pin, pout, qin, qout, rin, rout);
    __syncthreads();
    const bool readIn = alpha != T(0);
    const bool readOut = beta != T(0);
    if (readIn) {
        T v[M::NL][M::RL];
        M::load(in + rin, pin, qin, t, v);
        M::stash(tile, t, v);
    }
    __syncthreads();
    M::write(out + rout, pout, qout, tile, t, alpha, beta, readIn, readOut);
}

// Workgroups of the kernel resident on the device at once (looked up once
// per kernel and device, up to 64 devices; 0 when the runtime cannot say).
template <auto kernel>
unsigned resident(int threads)
{
    static std::atomic<int> cached[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 0;
    int n = dev >= 0 && dev < 64 ? cached[dev].load(std::memory_order_relaxed) : 0;
    if (n <= 0) {
        int cus = 0, per = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, kernel, threads, 0) != hipSuccess)
            return 0;
        n = cus * (per > 0 ? per : 1);
        if (dev >= 0 && dev < 64) cached[dev].store(n, std::memory_order_relaxed);
    }
    return (unsigned)n;
}

// P tiles per band when one row of P tiles would hold more than half of the
// resident workgroups (fp32 76832 x 2048 transposed: 4.9 TB/s walking
// P-fastest, 5.6 in bands of 32; no band width helps the other shapes)
constexpr int kBand = 32;

template <typename T, bool VL, bool VS, bool ALONGP>
hipError_t launch_t(unsigned blocks, hipStream_t s, TDesc d, const void *in, void *out,
                    double alpha, double beta)
{
    constexpr auto k = transpose_kernel<T, VL, VS, ALONGP>;
    const unsigned n = resident<k>(Shape<T>::TH);
    if (n == 0) return hipErrorInvalidValue;
    d.group = 2u * (unsigned)d.tiles[0] > n ? kBand : 0;
    hipLaunchKernelGGL(k, dim3(blocks), dim3(Shape<T>::TH), 0, s, d, static_cast<const T *>(in),
                       static_cast<T *>(out), (T)alpha, (T)beta);
    return hipGetLastError();
}

template <typename T>
hipError_t launch_typed(bool vl, bool vs, bool alongP, unsigned blocks, hipStream_t s,
                        const TDesc &d, const void *in, void *out, double alpha, double beta)
{
    auto go = [&](auto VLc, auto VSc) {
        return alongP ? launch_t<T, VLc.value, VSc.value, true>(blocks, s, d, in, out, alpha, beta)
                      : launch_t<T, VLc.value, VSc.value, false>(blocks, s, d, in, out, alpha, beta);
    };
    using Y = std::true_type;
    using N = std::false_type;
    if (vl && vs) return go(Y{}, Y{});
    if (vl) return go(Y{}, N{});
    if (vs) return go(N{}, Y{});
    return go(N{}, N{});
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
    const int kTP = dtype == GETT_FLOAT32 ? Shape<float>::TP : Shape<double>::TP;
    const int kTQ = dtype == GETT_FLOAT32 ? Shape<float>::TQ : Shape<double>::TQ;
    // P: by input stride until the tile edge is covered; Q: by output stride.
    // The output's stride-one index leads Q unless it is the input's too
    // (then the writes run along P): P takes no other index before it, or a
    // batched transposition such as (a,b,c,d) -> (b,a,d,c) would put b second
    // in P and write along P with a's output stride.
    std::vector<Idx> byIn = v, P, Q, R;
    std::stable_sort(byIn.begin(), byIn.end(), [](const Idx &a, const Idx &b) { return a.sin < b.sin; });
    size_t o1 = 0;
    for (size_t k = 1; k < byIn.size(); ++k)
        if (byIn[k].sout < byIn[o1].sout) o1 = k;
    int64_t sp = 1, sq = 1;
    std::vector<Idx> others;
    for (size_t k = 0; k < byIn.size(); ++k) {
        if (sp < kTP && (k != o1 || k == 0)) {
            P.push_back(byIn[k]);
            sp *= byIn[k].ext;
        } else {
            others.push_back(byIn[k]);
        }
    }
    std::stable_sort(others.begin(), others.end(), [](const Idx &a, const Idx &b) { return a.sout < b.sout; });
    size_t j = 0;
    for (; j < others.size() && sq < kTQ; ++j) {
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
    d.tiles[0] = (int32_t)((sp + kTP - 1) / kTP);
    d.tiles[1] = (int32_t)((sq + kTQ - 1) / kTQ);
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
    // 16-byte vectors: the run's first index is stride-one with an extent that
    // is a multiple of the vector, every other stride is a multiple of it, and
    // the base pointer is 16-byte aligned -- then no vector straddles an index
    // boundary or the end of a ragged tile, and every vector is aligned.
    const int vw = dtype == GETT_FLOAT32 ? 4 : 2;
    auto vec_ok = [&](const std::vector<Idx> &lead, bool inSide, const void *base) {
        if (lead.empty() || ((uintptr_t)base % 16)) return false;
        const Idx &f = lead[0];
        if ((inSide ? f.sin : f.sout) != 1 || f.ext % vw) return false;
        for (auto *g : {&P, &Q, &R})
            for (auto &x : *g)
                if (&x != &f && (inSide ? x.sin : x.sout) % vw) return false;
        return true;
    };
    const bool vl = alpha != 0.0 && vec_ok(P, true, in);
    const bool vs = vec_ok(d.alongP ? P : Q, false, out);
    const hipError_t e =
        dtype == GETT_FLOAT32
            ? launch_typed<float>(vl, vs, d.alongP != 0, (unsigned)blocks, stream, d, in, out, alpha,
                                  beta)
            : launch_typed<double>(vl, vs, d.alongP != 0, (unsigned)blocks, stream, d, in, out,
                                   alpha, beta);
    return e == hipSuccess ? GETT_SUCCESS : GETT_ERROR_HIP;
}

}  // namespace gett
