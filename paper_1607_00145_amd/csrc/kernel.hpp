// kernel.hpp -- the GETT macro-kernel for gfx950 (device code).
//
// One workgroup computes an MT x NT tile of the matrix view C[x][y]
// (Listing 4: the grid replaces the n- and m-loops (1) and (4); the in-kernel
// loop over K boxes is the k-loop (2)).  Per K box:
//   pack   -- X's MT x kbox sub-tensor and Y's NT x kbox sub-tensor are
//             gathered from device memory straight into LDS (Eq. 9-10: the
//             packing is a transposition into a fixed layout [k][row]); the
//             loads run along each operand's stride-one index;
//   macro  -- every wavefront multiplies its part of the packed tiles with
//             MFMA 16x16x4 instructions, accumulating in registers (the
//             register-resident C~ of Sec. 3.1);
// and after the last box
//   unpack -- C(x,y) <- alpha * acc + beta * C(x,y) through C's own strides
//             (Eq. 11); C is not read when beta == 0.
//
// Register tile of a wavefront.  Lane l (l16 = l % 16, g = l / 16) of an
// MFMA 16x16x4 supplies row l16 of the A-operand and column l16 of the
// B-operand at contracted position g, and receives four results of column
// l16 (rows Traits<T>::mrow(g, 0..3)).  One LDS read of R consecutive rows
// per lane feeds R blocks at once (R = RX on the row side, RY on the column
// side; 1, or VW = 16 bytes / element): within a group of 16*R rows, MFMA row
// r of block i is tile row R*r + i.  With RY = VW a lane owns VW consecutive
// columns of C for each of its rows, which the epilogue writes as one 16-byte
// vector; with the operands arranged so that C's stride-one index runs along
// y, 16 lanes store 256 contiguous bytes.  The contracted positions used by
// lane group g at MFMA step s are 4s + g for both operands, so each product
// pairs matching indices.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "desc.hpp"

namespace gett {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef double f64x2 __attribute__((ext_vector_type(2)));
typedef double f64x4 __attribute__((ext_vector_type(4)));

template <typename T> struct Traits;
// Result layout of the 16x16x4 MFMAs: lane l, accumulator element r holds
// row mrow(l / 16, r) of column l % 16.  The fp32 instruction gives each lane
// four consecutive rows; the fp64 instruction interleaves them with stride 4.
template <> struct Traits<float> {
    typedef f32x4 vec;   // 16-byte vector
    typedef f32x4 acc;   // 16x16 MFMA accumulator slice of one lane
    static constexpr int VW = 4;
    static __device__ __forceinline__ int mrow(int g, int r) { return 4 * g + r; }
};
template <> struct Traits<double> {
    typedef f64x2 vec;
    typedef f64x4 acc;
    static constexpr int VW = 2;
    static __device__ __forceinline__ int mrow(int g, int r) { return g + 4 * r; }
};

__device__ __forceinline__ f32x4 mfma16x16x4(float a, float b, f32x4 c)
{
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f64x4 mfma16x16x4(double a, double b, f64x4 c)
{
    return __builtin_amdgcn_mfma_f64_16x16x4f64(a, b, c, 0, 0, 0);
}

constexpr int kInvalidK = 0x7fffffff;

// Map the hardware workgroup id to a tile.  Workgroups are dealt round-robin
// to the 8 XCDs (each with its own L2); renumber so that consecutive logical
// tiles run on one XCD.  Then either walk tiles in bands of `group` x-tiles,
// so that neighbours share operand rows/columns in L2 (compute-bound
// contractions), or walk y fastest, so that the workgroups running at one time
// write neighbouring stretches of C (streaming contractions, where DRAM page
// locality of the C stream decides the bandwidth).
__device__ __forceinline__ void tile_of_block(const KDesc &d, int &tx, int &ty)
{
    const int nwg = (int)gridDim.x;
    const int bid = (int)blockIdx.x;
    const int full = nwg & ~7;
    int logical = bid;
    if (bid < full) logical = (bid & 7) * (full >> 3) + (bid >> 3);
    if (d.order == 1) {
        tx = logical / d.tilesY;
        ty = logical - tx * d.tilesY;
        return;
    }
    const int band = d.group * d.tilesY;
    const int first = (logical / band) * d.group;
    const int gsz = min(d.tilesX - first, d.group);
    const int in = logical - (logical / band) * band;
    tx = first + in % gsz;
    ty = in / gsz;
}

// Origin of K box `s`: block `s % nblk` of index kj, then one point of each
// later contracted index (first one fastest).  Returns the origin offsets in
// X and Y and the number of valid positions left along index kj.
__device__ __forceinline__ int box_origin(const KDesc &d, uint32_t s, int &ox, int &oy)
{
    const uint32_t nb = (uint32_t)d.nblk;
    const uint32_t rest0 = s / nb;
    const int blk = (int)(s - rest0 * nb);
    uint32_t rest = rest0;
    ox = blk * d.tj * (int)d.strXk[d.kj];
    oy = blk * d.tj * (int)d.strYk[d.kj];
    for (int i = d.kj + 1; i < d.nk; ++i) {
        const uint32_t e = (uint32_t)d.extK[i];
        const uint32_t q = rest / e;
        const uint32_t c = rest - q * e;
        rest = q;
        ox += (int)c * (int)d.strXk[i];
        oy += (int)c * (int)d.strYk[i];
    }
    return d.extK[d.kj] - blk * d.tj;
}

// Per-thread description of the part of one operand tile it gathers.  Item
// `it` of thread `tid` is element (or vector) tid + it * NTH of the tile in
// the mode's order; the tile shapes are chosen so that consecutive items of
// one thread are a fixed LDS distance apart.
template <typename T, int ROWS, int KT, int MODE, int NTH>
struct Gather {
    static constexpr int VW = Traits<T>::VW;
    static constexpr int PITCH = ROWS + VW;   // LDS row pitch (elements) of the [k][row] layout
    static constexpr int W = (MODE == kGatherScalar) ? 1 : VW;
    static constexpr int ITEMS = ROWS * KT / W;
    static constexpr int NI = ITEMS / NTH;
    static_assert(ITEMS % NTH == 0, "tile must split evenly over the workgroup");
    static_assert(NTH % (ROWS / VW) == 0 && NTH % (KT / VW) == 0 && NTH % KT == 0 &&
                      NTH % ROWS == 0,
                  "items of one thread must be a fixed LDS distance apart");
    typedef typename Traits<T>::vec vec;

    int goff[NI];   // element offset in the operand (without the box origin); < 2^31
    int kc[NI];     // position along index kj inside the box; kInvalidK: never valid
    int lds0;       // LDS slot of item 0
    int lstep;      // LDS distance between consecutive items
    T val[NI][W];   // staged values

    // rowoff: LDS table of operand offsets per tile row (-1 = outside the tensor)
    // koff/kco: LDS tables of offsets / kj-positions per box element
    __device__ __forceinline__ void setup(int tid, const int *rowoff, const int *koff,
                                          const int *kco, int kfast)
    {
#pragma unroll
        for (int it = 0; it < NI; ++it) {
            const int i = tid + it * NTH;
            int r, kk;
            if (MODE == kGatherRowVec) {
                r = (i % (ROWS / VW)) * VW;
                kk = i / (ROWS / VW);
            } else if (MODE == kGatherKVec) {
                kk = (i % (KT / VW)) * VW;
                r = i / (KT / VW);
            } else if (kfast) {
                kk = i % KT;
                r = i / KT;
            } else {
                r = i % ROWS;
                kk = i / ROWS;
            }
            const int ro = rowoff[r];
            goff[it] = (ro < 0 ? 0 : ro) + koff[kk];
            kc[it] = ro < 0 ? kInvalidK : kco[kk];
            if (it == 0) lds0 = kk * PITCH + r;
            if (it == 1) lstep = kk * PITCH + r - lds0;
        }
        if (NI == 1) lstep = 0;
    }

    __device__ __forceinline__ void load(const T *__restrict__ p, int limit)
    {
#pragma unroll
        for (int it = 0; it < NI; ++it) {
            if (kc[it] < limit) {
                if (W == 1) {
                    val[it][0] = p[goff[it]];
                } else {
                    const vec v = *reinterpret_cast<const vec *>(p + goff[it]);
#pragma unroll
                    for (int e = 0; e < W; ++e) val[it][e] = v[e];
                }
            } else {
#pragma unroll
                for (int e = 0; e < W; ++e) val[it][e] = T(0);
            }
        }
    }

    __device__ __forceinline__ void store(T *tile) const
    {
#pragma unroll
        for (int it = 0; it < NI; ++it) {
            T *dst = tile + lds0 + it * lstep;
            if (MODE == kGatherRowVec) {
                vec v;
#pragma unroll
                for (int e = 0; e < W; ++e) v[e] = val[it][e];
                *reinterpret_cast<vec *>(dst) = v;
            } else if (MODE == kGatherKVec) {
#pragma unroll
                for (int e = 0; e < W; ++e) dst[e * PITCH] = val[it][e];
            } else {
                *dst = val[it][0];
            }
        }
    }
};

// R consecutive elements read from LDS by one lane (R = 1: a scalar).
template <typename T, int R> struct RVec {
    typedef T __attribute__((ext_vector_type(R))) type;
    static __device__ __forceinline__ T at(const type &v, int i) { return v[i]; }
};
template <typename T> struct RVec<T, 1> {
    typedef T type;
    static __device__ __forceinline__ T at(const type &v, int) { return v; }
};

// Tile row of MFMA row `rho` in block `b` when R rows are read per lane.
template <int R> __device__ __forceinline__ int block_row(int b, int rho)
{
    return (b / R) * 16 * R + R * rho + (b % R);
}

template <typename T, int MT, int NT, int KT, int WM, int WN, int RX, int RY, int WPE, int XMODE,
          int YMODE>
__global__ void __launch_bounds__(WM *WN * 64) __attribute__((amdgpu_waves_per_eu(WPE)))
gett_macro_kernel(const KDesc d, const T *__restrict__ X, const T *__restrict__ Y,
                  T *__restrict__ C, const T alpha, const T beta)
{
    constexpr int NTH = WM * WN * 64;
    constexpr int VW = Traits<T>::VW;
    constexpr int WTM = MT / WM;            // wave tile rows
    constexpr int WTN = NT / WN;            // wave tile columns
    constexpr int RB = WTM / 16;            // MFMA blocks per wave along x
    constexpr int CB = WTN / 16;            // MFMA blocks per wave along y
    static_assert(WTM % (16 * RX) == 0 && WTN % (16 * RY) == 0,
                  "wave tile must be a multiple of 16*R in both directions");
    static_assert(RX == 1 || RX == 2 || RX == 4, "read width");
    static_assert(RY == 1 || RY == 2 || RY == 4, "read width");
    static_assert(RX <= VW && RY <= VW, "at most 16 bytes per LDS read");
    static_assert(KT % 4 == 0, "K tile must be a multiple of the MFMA depth");
    typedef Gather<T, MT, KT, XMODE, NTH> GX;
    typedef Gather<T, NT, KT, YMODE, NTH> GY;
    typedef typename Traits<T>::vec vec;
    typedef typename Traits<T>::acc accv;
    typedef RVec<T, RX> XV;
    typedef RVec<T, RY> YV;

    __shared__ __attribute__((aligned(16))) T xs[2][KT * GX::PITCH];
    __shared__ __attribute__((aligned(16))) T ys[2][KT * GY::PITCH];
    // Element offsets fit in 31 bits (the plan refuses larger tensors); -1 marks
    // a row or column outside the tensor.
    __shared__ int rowX[MT], rowY[NT], offCx[MT], offCy[NT];
    __shared__ int kX[KT], kY[KT];
    __shared__ int kco[KT];

    const int tid = (int)threadIdx.x;
    int tx, ty;
    tile_of_block(d, tx, ty);

    // ---- identify_subtensor: offsets of this tile's rows, columns, box ----
    for (int r = tid; r < MT; r += NTH) {
        uint32_t x = (uint32_t)tx * MT + r;
        int ox = -1, oc = -1;
        if ((int64_t)x < d.sizeX) {
            ox = 0;
            oc = 0;
            for (int i = 0; i < d.nx; ++i) {
                const uint32_t e = (uint32_t)d.extX[i];
                const uint32_t q = x / e;
                const uint32_t id = x - q * e;
                x = q;
                ox += (int)id * (int)d.strXop[i];
                oc += (int)id * (int)d.strCx[i];
            }
        }
        rowX[r] = ox;
        offCx[r] = oc;
    }
    for (int r = tid; r < NT; r += NTH) {
        uint32_t y = (uint32_t)ty * NT + r;
        int oy = -1, oc = -1;
        if ((int64_t)y < d.sizeY) {
            oy = 0;
            oc = 0;
            for (int i = 0; i < d.ny; ++i) {
                const uint32_t e = (uint32_t)d.extY[i];
                const uint32_t q = y / e;
                const uint32_t id = y - q * e;
                y = q;
                oy += (int)id * (int)d.strYop[i];
                oc += (int)id * (int)d.strCy[i];
            }
        }
        rowY[r] = oy;
        offCy[r] = oc;
    }
    for (int kk = tid; kk < KT; kk += NTH) {
        int ox = 0, oy = 0;
        int pos = kInvalidK;
        if (kk < d.kbox) {
            uint32_t k = (uint32_t)kk;
            for (int i = 0; i < d.kj; ++i) {
                const uint32_t e = (uint32_t)d.extK[i];
                const uint32_t q = k / e;
                const uint32_t id = k - q * e;
                k = q;
                ox += (int)id * (int)d.strXk[i];
                oy += (int)id * (int)d.strYk[i];
            }
            pos = (int)k;   // position along index kj, < tj
            ox += (int)k * (int)d.strXk[d.kj];
            oy += (int)k * (int)d.strYk[d.kj];
        }
        kX[kk] = ox;
        kY[kk] = oy;
        kco[kk] = pos;
    }
    __syncthreads();

    GX gx;
    GY gy;
    gx.setup(tid, rowX, kX, kco, d.xscalar_kfast);
    gy.setup(tid, rowY, kY, kco, d.yscalar_kfast);

    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wm = wave % WM;
    const int wn = wave / WM;
    const int l16 = lane & 15;
    const int g = lane >> 4;

    accv acc[RB][CB];
#pragma unroll
    for (int a = 0; a < RB; ++a)
#pragma unroll
        for (int b = 0; b < CB; ++b)
#pragma unroll
            for (int r = 0; r < 4; ++r) acc[a][b][r] = T(0);

    // The lane's C rows, RX blocks (4*RX rows) at a time, and its columns.
    constexpr int NR = 4 * RX;
    auto rows_of = [&](int grp, int *ox) {
#pragma unroll
        for (int i = 0; i < RX; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r)
                ox[i * 4 + r] =
                    offCx[wm * WTM + block_row<RX>(grp * RX + i, Traits<T>::mrow(g, r))];
    };
    // With RY == VW and C vectors enabled, column group cg's VW columns are
    // consecutive: one offset per group.
    constexpr bool kVecC = RY == VW;
    constexpr int CGV = CB / RY;   // column groups per wave
    auto cols_of = [&](int *oy) {
#pragma unroll
        for (int cg = 0; cg < CGV; ++cg) oy[cg] = offCy[wn * WTN + cg * 16 * RY + RY * l16];
    };
    const bool readC = beta != T(0);
    const bool useCvec = kVecC && d.cvec;
    const uint32_t nsteps = (uint32_t)d.nsteps;
    if (nsteps > 0) {
        int ox, oy;
        const int lim = box_origin(d, 0, ox, oy);
        gx.load(X + ox, lim);
        gy.load(Y + oy, lim);
        gx.store(xs[0]);
        gy.store(ys[0]);
    }
    __syncthreads();

    for (uint32_t s = 0; s < nsteps; ++s) {
        const int buf = (int)(s & 1);
        const bool more = s + 1 < nsteps;
        if (more) {
            int ox, oy;
            const int lim = box_origin(d, s + 1, ox, oy);
            gx.load(X + ox, lim);
            gy.load(Y + oy, lim);
        }
        const T *xt = xs[buf] + wm * WTM + RX * l16;
        const T *yt = ys[buf] + wn * WTN + RY * l16;
#pragma unroll
        for (int ks = 0; ks < KT / 4; ++ks) {
            const int k = 4 * ks + g;
            typename XV::type av[RB / RX];
            typename YV::type bv[CB / RY];
#pragma unroll
            for (int gi = 0; gi < RB / RX; ++gi)
                av[gi] = *reinterpret_cast<const typename XV::type *>(xt + k * GX::PITCH + gi * 16 * RX);
#pragma unroll
            for (int gj = 0; gj < CB / RY; ++gj)
                bv[gj] = *reinterpret_cast<const typename YV::type *>(yt + k * GY::PITCH + gj * 16 * RY);
#pragma unroll
            for (int a = 0; a < RB; ++a)
#pragma unroll
                for (int b = 0; b < CB; ++b)
                    acc[a][b] = mfma16x16x4(XV::at(av[a / RX], a % RX), YV::at(bv[b / RY], b % RY),
                                            acc[a][b]);
        }
        if (more) {
            gx.store(xs[buf ^ 1]);
            gy.store(ys[buf ^ 1]);
        }
        __syncthreads();
    }

    // ---- unpack: C <- alpha * acc + beta * C through C's strides (Eq. 11) ----
    // RX blocks of rows at a time: first every C load of the group (so they are
    // in flight together), then the updates and non-temporal stores (C is
    // written once and not reused).
#pragma unroll
    for (int grp = 0; grp < RB / RX; ++grp) {
        int ox[NR];
        rows_of(grp, ox);
        if (useCvec) {
            int oy[CGV];
            cols_of(oy);
            vec cv[NR][CGV];
            if (readC) {
#pragma unroll
                for (int q = 0; q < NR; ++q)
#pragma unroll
                    for (int cg = 0; cg < CGV; ++cg)
                        if (ox[q] >= 0 && oy[cg] >= 0)
                            cv[q][cg] = __builtin_nontemporal_load(
                                reinterpret_cast<const vec *>(C + ox[q] + oy[cg]));
            }
#pragma unroll
            for (int q = 0; q < NR; ++q)
#pragma unroll
                for (int cg = 0; cg < CGV; ++cg) {
                    if (ox[q] < 0 || oy[cg] < 0) continue;
                    vec out;
#pragma unroll
                    for (int j = 0; j < VW; ++j) {
                        const T a = alpha * acc[grp * RX + q / 4][kVecC ? cg * RY + j : 0][q % 4];
                        out[j] = readC ? a + beta * cv[q][cg][j] : a;
                    }
                    __builtin_nontemporal_store(out, reinterpret_cast<vec *>(C + ox[q] + oy[cg]));
                }
        } else {
            int oy[CB];
#pragma unroll
            for (int b = 0; b < CB; ++b) oy[b] = offCy[wn * WTN + block_row<RY>(b, l16)];
            T cv[NR][CB];
            if (readC) {
#pragma unroll
                for (int q = 0; q < NR; ++q)
#pragma unroll
                    for (int b = 0; b < CB; ++b)
                        if (ox[q] >= 0 && oy[b] >= 0)
                            cv[q][b] = __builtin_nontemporal_load(C + ox[q] + oy[b]);
            }
#pragma unroll
            for (int q = 0; q < NR; ++q)
#pragma unroll
                for (int b = 0; b < CB; ++b) {
                    if (ox[q] < 0 || oy[b] < 0) continue;
                    const T a = alpha * acc[grp * RX + q / 4][b][q % 4];
                    __builtin_nontemporal_store(readC ? a + beta * cv[q][b] : a, C + ox[q] + oy[b]);
                }
        }
    }
}

}  // namespace gett
