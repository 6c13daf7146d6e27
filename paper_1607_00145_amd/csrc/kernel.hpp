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

#include <type_traits>

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

// s_waitcnt operand that waits for every vector memory operation of the
// wavefront to complete (vmcnt 0) and leaves the other counters alone
// (expcnt 7, lgkmcnt 15; gfx9 encoding).
constexpr int kWaitStores = (7 << 4) | (15 << 8);

// Map the hardware workgroup id to a tile.  Workgroups are dealt round-robin
// to the 8 XCDs (each with its own L2); renumber so that consecutive logical
// tiles run on one XCD.  Then either walk tiles in bands of `group` x-tiles,
// so that neighbours share operand rows/columns in L2 (compute-bound
// contractions), or walk y fastest, so that the workgroups running at one time
// write neighbouring stretches of C (streaming contractions, where DRAM page
// locality of the C stream decides the bandwidth).
__device__ __forceinline__ void tile_of_block(const KDesc &d, int bid, int nwg, int &tx, int &ty)
{
    const int full = nwg & ~7;
    int logical = bid;
    if (d.xcdremap && bid < full) logical = (bid & 7) * (full >> 3) + (bid >> 3);
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
// X and Y (64-bit: a tensor may hold 2^31 elements or more) and the number of
// valid positions left along index kj.
__device__ __forceinline__ int box_origin(const KDesc &d, uint32_t s, int64_t &ox, int64_t &oy)
{
    const uint32_t nb = (uint32_t)d.nblk;
    const uint32_t rest0 = s / nb;
    const int blk = (int)(s - rest0 * nb);
    uint32_t rest = rest0;
    ox = (int64_t)(blk * d.tj) * d.strXk[d.kj];
    oy = (int64_t)(blk * d.tj) * d.strYk[d.kj];
    for (int i = d.kj + 1; i < d.nk; ++i) {
        const uint32_t e = (uint32_t)d.extK[i];
        const uint32_t q = rest / e;
        const uint32_t c = rest - q * e;
        rest = q;
        ox += (int64_t)c * d.strXk[i];
        oy += (int64_t)c * d.strYk[i];
    }
    return d.extK[d.kj] - blk * d.tj;
}

// Origins of consecutive K boxes without a division per box: the block
// along index kj advances by one; when it wraps, the first later contracted
// index advances (extent and strides held in registers), and only when that
// one wraps too is the origin decomposed afresh by box_origin.  Any box may
// be asked for; consecutive ones cost a few scalar additions.
struct BoxWalker {
    uint32_t cur;        // box whose origin is held
    int64_t ox, oy;      // its origins in X and Y
    int lim;             // valid positions along kj
    int blk, c1;         // its block along kj and value of index kj + 1
    int nblk, e1;        // blocks along kj; extent of index kj + 1 (0: none)
    int64_t bx, by;      // origin step of one block along kj in X and Y
    int64_t sx1, sy1;    // strides of index kj + 1 in X and Y
    int ek, tj;          // extent of index kj and its block length

    __device__ __forceinline__ void reset(const KDesc &d, uint32_t s)
    {
        cur = s;
        lim = box_origin(d, s, ox, oy);
        blk = (int)(s % (uint32_t)nblk);
        c1 = e1 > 0 ? (int)((s / (uint32_t)nblk) % (uint32_t)e1) : 0;
    }
    __device__ __forceinline__ void init(const KDesc &d, uint32_t s)
    {
        nblk = d.nblk > 0 ? d.nblk : 1;
        tj = d.tj;
        ek = d.extK[d.kj];
        bx = (int64_t)d.tj * d.strXk[d.kj];
        by = (int64_t)d.tj * d.strYk[d.kj];
        const bool later = d.kj + 1 < d.nk;
        e1 = later ? d.extK[d.kj + 1] : 0;
        sx1 = later ? d.strXk[d.kj + 1] : 0;
        sy1 = later ? d.strYk[d.kj + 1] : 0;
        reset(d, s);
    }
    // origin of box s (returns the valid positions along kj)
    __device__ __forceinline__ int at(const KDesc &d, uint32_t s, int64_t &x, int64_t &y)
    {
        if (s == cur + 1) {
            cur = s;
            if (++blk < nblk) {
                ox += bx;
                oy += by;
                lim -= tj;
            } else if (++c1 < e1) {
                blk = 0;
                ox += sx1 - (int64_t)(nblk - 1) * bx;
                oy += sy1 - (int64_t)(nblk - 1) * by;
                lim = ek;
            } else {
                reset(d, s);
            }
        } else if (s != cur) {
            reset(d, s);
        }
        x = ox;
        y = oy;
        return lim;
    }
};

// Per-thread description of the part of one operand tile it gathers.  Item
// `it` of thread `tid` is element (or 16-byte vector) tid + it * NTH of the
// tile in the mode's order; items past the tile's end are idle.
//
// The strided modes gather a tile whose rows (or K positions) are ordered
// (u, v, ...) with u of extent `es` fastest and the operand's stride-one index
// v second: the VW elements of one vector are es rows (K positions) apart in
// the packed layout and are written to LDS one by one.  Within a line of
// ROWS rows (KT positions) an item is (q, c): vector q along v (fastest, so
// that neighbouring lanes read neighbouring 16-byte pieces) at u = c; the
// analyser guarantees es * VW divides ROWS (KT) and that v's extent and, in
// the K box, its block length are multiples of VW, so a vector is valid or
// outside the tensor as a whole.
template <typename T, int ROWS, int KT, int MODE, int NTH, int STAGES = 1, bool SWZ = false>
struct Gather {
    static constexpr int VW = Traits<T>::VW;
    static constexpr int PITCH = ROWS + VW;   // LDS row pitch (elements) of the [k][row] layout
    static constexpr bool kRowV = MODE == kGatherRowVec || MODE == kGatherRowVecStrided;
    static constexpr bool kKV = MODE == kGatherKVec || MODE == kGatherKVecStrided;
    static constexpr bool kStrided = MODE == kGatherRowVecStrided || MODE == kGatherKVecStrided;
    static constexpr int W = (MODE == kGatherScalar) ? 1 : VW;
    static_assert(MODE == kGatherScalar || (ROWS % VW == 0 && KT % VW == 0), "vector gathers");
    static constexpr int ITEMS = ROWS * KT / W;
    static constexpr int NI = (ITEMS + NTH - 1) / NTH;
    static constexpr bool kFull = ITEMS % NTH == 0;
    // Swizzle of the k-vector gather: the VW elements of a vector go to VW
    // LDS lines (one per contracted position), all at one row; without it
    // the lines of the vectors a wavefront stores start at two banks only
    // (the pitch is ROWS + VW), so these stores conflict 4-way.  Row r of
    // line k is stored at row swz(r, k) = r ^ (VW * ((k / 4) mod 8)): lines
    // of different groups of four shift by whole vectors, a vector's VW
    // elements share the shift (VW divides 4), and a VW-row piece stays
    // contiguous for the MFMA reads, which apply the same bijection (for the
    // rows of one MFMA step the shift is a constant).  SWZ: the kernel asks
    // for it only when the other operand is gathered in vectors too; beside
    // an element-wise or strided gather, whose addressing already fills the
    // register budget, the swizzled reads made the compiler spill (64 x 256
    // fp32 tile: 0 -> 176 bytes per lane, twice the time).
    static constexpr bool kSwz = SWZ && MODE == kGatherKVec && ROWS % (8 * VW) == 0;
    static __device__ __forceinline__ int swz(int r, int k)
    {
        return kSwz ? r ^ (VW * ((k >> 2) & 7)) : r;
    }
    // Consecutive items of one thread sit a fixed LDS distance apart when the
    // workgroup covers whole rows (or whole K lines) per item round (and, with
    // the swizzle, the rows of one round are a multiple of the shifted span).
    static constexpr bool kConst =
        NI <= 1 || (kFull && (kRowV ? NTH % (ROWS / VW) == 0
                              : kKV ? NTH % (KT / VW) == 0 &&
                                          (!kSwz || (NTH / (KT / VW)) % (8 * VW) == 0)
                                    : NTH % KT == 0 && NTH % ROWS == 0));
    typedef typename Traits<T>::vec vec;

    int goff[NI];                 // element offset in the operand (without the box origin)
    int kc[NI];                   // position along index kj inside the box; kInvalidK: never valid
    int lds[kConst ? 1 : NI];     // LDS slot of each item (of item 0 when kConst); -1: idle
    int lstep;                    // LDS distance between consecutive items (kConst)
    int estep;                    // LDS distance between the elements of a strided vector
    T val[STAGES][NI][W];         // staged values, one set per stage in flight

    // rowoff: LDS table of operand offsets per tile row (-1 = outside the tensor)
    // koff/kco: LDS tables of offsets / kj-positions per box element
    // es: extent of the first row (K) index in the strided modes
    // perm (scalar rows-fastest mode only, may be null): lane order over the
    // tile rows -- item row r gathers tile row perm[r]
    __device__ __forceinline__ void setup(int tid, const int *rowoff, const int *koff,
                                          const int *kco, int kfast, int es = 1,
                                          const int *perm = nullptr)
    {
        lstep = 0;
        estep = MODE == kGatherKVecStrided ? es * PITCH : es;
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
            } else if (MODE == kGatherRowVecStrided) {
                const int j = i % (ROWS / VW), nq = ROWS / (VW * es);
                r = (j / nq) + (j % nq) * es * VW;
                kk = i / (ROWS / VW);
            } else if (MODE == kGatherKVecStrided) {
                const int j = i % (KT / VW), nq = KT / (VW * es);
                kk = (j / nq) + (j % nq) * es * VW;
                r = i / (KT / VW);
            } else if (kfast) {
                kk = i % KT;
                r = i / KT;
            } else {
                r = i % ROWS;
                kk = i / ROWS;
                if (perm) r = perm[r];
            }
            const bool act = kFull || i < ITEMS;
            const int ro = act ? rowoff[r] : -1;
            goff[it] = (ro < 0 ? 0 : ro) + (act ? koff[kk] : 0);
            kc[it] = ro < 0 ? kInvalidK : kco[kk];
            const int slot = act ? kk * PITCH + swz(r, kk) : -1;
            if (kConst) {
                if (it == 0) lds[0] = slot;
                if (it == 1) lstep = slot - lds[0];
            } else {
                lds[kConst ? 0 : it] = slot;
            }
        }
    }

    template <int B = 0>
    __device__ __forceinline__ void load(const T *__restrict__ p, int limit)
    {
#pragma unroll
        for (int it = 0; it < NI; ++it) {
            if (kc[it] < limit) {
                if (W == 1) {
                    val[B][it][0] = p[goff[it]];
                } else {
                    const vec v = *reinterpret_cast<const vec *>(p + goff[it]);
#pragma unroll
                    for (int e = 0; e < W; ++e) val[B][it][e] = v[e];
                }
            } else {
#pragma unroll
                for (int e = 0; e < W; ++e) val[B][it][e] = T(0);
            }
        }
    }

    // load(p, limit) then store(tile), one item at a time (few registers)
    __device__ __forceinline__ void copy(const T *__restrict__ p, int limit, T *tile)
    {
#pragma unroll
        for (int it = 0; it < NI; ++it) {
            const int slot = kConst ? lds[0] + it * lstep : lds[kConst ? 0 : it];
            if (!kFull && slot < 0) continue;
            T v[W];
            if (kc[it] < limit) {
                if (W == 1) {
                    v[0] = p[goff[it]];
                } else {
                    const vec x = *reinterpret_cast<const vec *>(p + goff[it]);
#pragma unroll
                    for (int e = 0; e < W; ++e) v[e] = x[e];
                }
            } else {
#pragma unroll
                for (int e = 0; e < W; ++e) v[e] = T(0);
            }
            T *dst = tile + slot;
            if (MODE == kGatherRowVec) {
                vec x;
#pragma unroll
                for (int e = 0; e < W; ++e) x[e] = v[e];
                *reinterpret_cast<vec *>(dst) = x;
            } else if (MODE == kGatherKVec) {
#pragma unroll
                for (int e = 0; e < W; ++e) dst[e * PITCH] = v[e];
            } else if (kStrided) {
#pragma unroll
                for (int e = 0; e < W; ++e) dst[e * estep] = v[e];
            } else {
                *dst = v[0];
            }
        }
    }

    template <int B = 0>
    __device__ __forceinline__ void store(T *tile) const
    {
#pragma unroll
        for (int it = 0; it < NI; ++it) {
            const int slot = kConst ? lds[0] + it * lstep : lds[kConst ? 0 : it];
            if (!kFull && slot < 0) continue;
            T *dst = tile + slot;
            if (MODE == kGatherRowVec) {
                vec v;
#pragma unroll
                for (int e = 0; e < W; ++e) v[e] = val[B][it][e];
                *reinterpret_cast<vec *>(dst) = v;
            } else if (MODE == kGatherKVec) {
#pragma unroll
                for (int e = 0; e < W; ++e) dst[e * PITCH] = val[B][it][e];
            } else if (kStrided) {
#pragma unroll
                for (int e = 0; e < W; ++e) dst[e * estep] = val[B][it][e];
            } else {
                *dst = val[B][it][0];
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

// Lowest offset any of the positions [x0, x1] of a linearised set can have
// (in the operand and in C), taken digit by digit: a digit that wraps inside
// the range can be 0, one that does not keeps its value at x0.  Offsets of the
// range relative to it are then >= 0, and the analyser bounds them by 2^31 - 1
// (the tile's own span), so the per-tile tables hold 32-bit offsets while the
// tensors may be larger.
__device__ __forceinline__ void range_base(int n, const int32_t *ext, const int64_t *sop,
                                           const int64_t *sc, uint32_t x0, uint32_t x1,
                                           int64_t &bop, int64_t &bc)
{
    bop = 0;
    bc = 0;
    for (int i = 0; i < n; ++i) {
        const uint32_t e = (uint32_t)ext[i];
        const uint32_t q0 = x0 / e, q1 = x1 / e;
        const int64_t dmin = q0 == q1 ? (int64_t)(x0 - q0 * e) : 0;
        bop += dmin * sop[i];
        bc += dmin * sc[i];
        x0 = q0;
        x1 = q1;
    }
}

// A value the whole wavefront shares, said so to the compiler (it then stays
// in scalar registers: a C base it takes for a per-lane value costs the
// epilogue its batched loads -- each load of C followed by its own wait).
__device__ __forceinline__ int uniform(int v) { return __builtin_amdgcn_readfirstlane(v); }
__device__ __forceinline__ int64_t uniform(int64_t v)
{
    const uint32_t lo = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)v);
    const uint32_t hi = (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)(v >> 32));
    return (int64_t)(((uint64_t)hi << 32) | lo);
}

// Base offsets of one tile: rows [tx MT, ...) of the x set, columns
// [ty NT, ...) of the y set, in the operands and in C.
struct TileBase {
    int64_t x, cx, y, cy;
};

template <int MT, int NT>
__device__ __forceinline__ TileBase tile_base(const KDesc &d, int tx, int ty)
{
    TileBase b;
    const uint32_t x0 = (uint32_t)(uniform(tx) * MT), y0 = (uint32_t)(uniform(ty) * NT);
    const uint32_t x1 = (uint32_t)min((int64_t)x0 + MT, d.sizeX) - 1;
    const uint32_t y1 = (uint32_t)min((int64_t)y0 + NT, d.sizeY) - 1;
    range_base(d.nx, d.extX, d.strXop, d.strCx, x0, x1, b.x, b.cx);
    range_base(d.ny, d.extY, d.strYop, d.strCy, y0, y1, b.y, b.cy);
    b.x = uniform(b.x);
    b.cx = uniform(b.cx);
    b.y = uniform(b.y);
    b.cy = uniform(b.cy);
    return b;
}

// identify_subtensor for one tile: operand and C offsets of every tile row
// (x side) and column (y side), relative to the tile's base offsets, one
// mixed-radix decomposition each.
template <int MT, int NT, int NTH>
__device__ __forceinline__ void tile_tables(const KDesc &d, int tx, int ty, const TileBase &b,
                                            int tid, int *rowX, int *offCx, int *rowY, int *offCy)
{
    // the x and y sides in separate branches: each reads its descriptor
    // arrays at wave-uniform indices (scalar loads, which do not wait behind
    // the wavefront's vector memory instructions in flight)
    auto decode = [](uint32_t v, int n, const int32_t *ext, const int64_t *so, const int64_t *sc,
                     int64_t &o64, int64_t &c64) {
        o64 = 0;
        c64 = 0;
        for (int i = 0; i < n; ++i) {
            const uint32_t e = (uint32_t)ext[i];
            const uint32_t q = v / e;
            const uint32_t id = v - q * e;
            v = q;
            o64 += (int64_t)id * so[i];
            c64 += (int64_t)id * sc[i];
        }
    };
    for (int r = tid; r < MT + NT; r += NTH) {
        int64_t o64, c64;
        if (r < MT) {
            const uint32_t v = (uint32_t)(tx * MT) + r;
            int oo = -1, oc = -1;
            if ((int64_t)v < d.sizeX) {
                decode(v, d.nx, d.extX, d.strXop, d.strCx, o64, c64);
                oo = (int)(o64 - b.x);
                oc = (int)(c64 - b.cx);
            }
            rowX[r] = oo;
            offCx[r] = oc;
        } else {
            const int rr = r - MT;
            const uint32_t v = (uint32_t)(ty * NT) + rr;
            int oo = -1, oc = -1;
            if ((int64_t)v < d.sizeY) {
                decode(v, d.ny, d.extY, d.strYop, d.strCy, o64, c64);
                oo = (int)(o64 - b.y);
                oc = (int)(c64 - b.cy);
            }
            rowY[rr] = oo;
            offCy[rr] = oc;
        }
    }
}

// Offsets and kj-positions of the positions of one K box.
template <int KT, int NTH>
__device__ __forceinline__ void box_tables(const KDesc &d, int tid, int *kX, int *kY, int *kco)
{
    for (int kk = tid; kk < KT; kk += NTH) {
        int ox = 0, oy = 0;
        int pos = kInvalidK;
        if (kk < d.kbox) {
            uint32_t k = (uint32_t)kk;
            int64_t x64 = 0, y64 = 0;
            for (int i = 0; i < d.kj; ++i) {
                const uint32_t e = (uint32_t)d.extK[i];
                const uint32_t q = k / e;
                const uint32_t id = k - q * e;
                k = q;
                x64 += (int64_t)id * d.strXk[i];
                y64 += (int64_t)id * d.strYk[i];
            }
            pos = (int)k;   // position along index kj, < tj
            x64 += (int64_t)k * d.strXk[d.kj];
            y64 += (int64_t)k * d.strYk[d.kj];
            // within the box's span, which the analyser bounds by 2^31 - 1
            ox = (int)x64;
            oy = (int)y64;
        }
        kX[kk] = ox;
        kY[kk] = oy;
        kco[kk] = pos;
    }
}

// Lane order for an element-wise gather whose operand is stride-one along
// the second index of the tile's rows (the first, of extent E, has a large
// stride there): rows are taken grouped by y mod E and then by y / E, so that
// consecutive lanes step along the operand's stride-one index.  Row r of the
// tile (global y = y0 + r) goes to position
//   start(a) + (r - t(a)) / E,   a = y mod E, t(a) = (a - y0) mod E,
// where start(a) counts the rows of the residues before a: each residue has
// q = R / E rows plus one if t < R mod E.
template <int R, int NTH>
__device__ __forceinline__ void row_perm(int E, int y0, int tid, int *perm)
{
    const int q = R / E, rem = R % E, s = y0 % E;
    const int u = (E - s) % E;   // t of residue 0
    for (int r = tid; r < R; r += NTH) {
        const int a = (y0 + r) % E;
        const int t = (a - s + E) % E;
        // residues 0..a-1 have t in the cyclic range [u, u + a) mod E; count those below rem
        int below;
        if (u + a <= E) {
            below = max(0, min(u + a, rem) - u);
        } else {
            below = max(0, rem - u) + min(u + a - E, rem);
        }
        perm[a * q + below + (r - t) / E] = r;
    }
}

// The register tile of one wavefront and the operations on it.
template <typename T, int MT, int NT, int KT, int WM, int WN, int RX, int RY>
struct WaveTile {
    static constexpr int VW = Traits<T>::VW;
    static constexpr int WTM = MT / WM;   // wave tile rows
    static constexpr int WTN = NT / WN;   // wave tile columns
    static constexpr int RB = WTM / 16;   // MFMA blocks per wave along x
    static constexpr int CB = WTN / 16;   // MFMA blocks per wave along y
    static_assert(WTM % (16 * RX) == 0 && WTN % (16 * RY) == 0,
                  "wave tile must be a multiple of 16*R in both directions");
    static_assert(RX == 1 || RX == 2 || RX == 4, "read width");
    static_assert(RY == 1 || RY == 2 || RY == 4, "read width");
    static_assert(RX <= VW && RY <= VW, "at most 16 bytes per LDS read");
    static_assert(KT % 4 == 0, "K tile must be a multiple of the MFMA depth");
    static constexpr int NR = 4 * RX;       // rows of one epilogue group owned by a lane
    static constexpr bool kVecC = RY == VW; // a lane owns VW consecutive columns
    static constexpr int CGV = CB / RY;     // column groups per wave
    typedef typename Traits<T>::vec vec;
    typedef typename Traits<T>::acc accv;
    typedef RVec<T, RX> XV;
    typedef RVec<T, RY> YV;

    accv acc[RB][CB];
    int wm, wn, l16, g;

    __device__ __forceinline__ void init(int tid)
    {
        const int lane = tid & 63;
        const int wave = tid >> 6;
        wm = wave % WM;
        wn = wave / WM;
        l16 = lane & 15;
        g = lane >> 4;
    }

    __device__ __forceinline__ void zero()
    {
#pragma unroll
        for (int a = 0; a < RB; ++a)
#pragma unroll
            for (int b = 0; b < CB; ++b)
#pragma unroll
                for (int r = 0; r < 4; ++r) acc[a][b][r] = T(0);
    }

    // acc += X~ * Y~ over the KT positions of one packed box (LDS [k][row]);
    // FIRST: acc = X~ * Y~ (the accumulators need no zeroing beforehand).
    // KU > 0 unrolls the MFMA steps KU at a time, which bounds how many LDS
    // reads the compiler hoists ahead of the MFMAs (registers).
    // PIPE: the fragments of step ks + 1 are read into a second register set
    // while the MFMAs of step ks are issued (scheduling groups interleave
    // them), so one wavefront alone on its SIMD does not wait for LDS between
    // steps.
    // SX / SY: the panel was stored with the k-vector swizzle (Gather::swz):
    // row r of line k sits at r ^ (VW * ((k / 4) mod 8)); the lines of MFMA
    // step ks are 4 ks .. 4 ks + 3, so the shift of a step is VW * (ks mod 8).
    template <int PX, int PY, bool FIRST = false, int KU = 0, bool PIPE = false, bool SX = false,
              bool SY = false>
    __device__ __forceinline__ void macro(const T *xs, const T *ys)
    {
        // Fragment gi of this lane starts at row w + RX * l16 + 16 RX gi of the
        // panel (w: the wave's first row, a multiple of 16 RX).  With the
        // swizzle a step's rows are XORed with c = VW * (ks mod 8).  When c is
        // below the block stride 16 RX (a power of two), the XOR touches only
        // the bits of RX * l16 and leaves w + 16 RX gi alone, so one XOR per
        // step serves every block and the block offset stays an immediate;
        // otherwise (tiles with RX = 1) the whole row is XORed.
        const int xw = wm * WTM, yw = wn * WTN, xl = RX * l16, yl = RY * l16;
        const T *xt = xs + xw + xl, *yt = ys + yw + yl;
        auto xat = [&](int ks, int k, int gi) {
            if constexpr (!SX) return xt + k * PX + gi * 16 * RX;
            else if constexpr (8 * VW <= 16 * RX)
                return xs + xw + k * PX + gi * 16 * RX + (xl ^ (VW * (ks & 7)));
            else return xs + k * PX + ((xw + xl + gi * 16 * RX) ^ (VW * (ks & 7)));
        };
        auto yat = [&](int ks, int k, int gj) {
            if constexpr (!SY) return yt + k * PY + gj * 16 * RY;
            else if constexpr (8 * VW <= 16 * RY)
                return ys + yw + k * PY + gj * 16 * RY + (yl ^ (VW * (ks & 7)));
            else return ys + k * PY + ((yw + yl + gj * 16 * RY) ^ (VW * (ks & 7)));
        };
        if constexpr (PIPE) {
            typename XV::type av[2][RB / RX];
            typename YV::type bv[2][CB / RY];
            auto read = [&](int ks, int buf) {
                const int k = 4 * ks + g;
#pragma unroll
                for (int gi = 0; gi < RB / RX; ++gi)
                    av[buf][gi] = *reinterpret_cast<const typename XV::type *>(xat(ks, k, gi));
#pragma unroll
                for (int gj = 0; gj < CB / RY; ++gj)
                    bv[buf][gj] = *reinterpret_cast<const typename YV::type *>(yat(ks, k, gj));
            };
            constexpr int NREAD = RB / RX + CB / RY;   // LDS reads per step
            constexpr int NMFMA = RB * CB;             // MFMAs per step
            read(0, 0);
#pragma unroll
            for (int ks = 0; ks < KT / 4; ++ks) {
                if (ks + 1 < KT / 4) read(ks + 1, (ks + 1) & 1);
#pragma unroll
                for (int a = 0; a < RB; ++a)
#pragma unroll
                    for (int b = 0; b < CB; ++b)
                        acc[a][b] = mfma16x16x4(XV::at(av[ks & 1][a / RX], a % RX),
                                                YV::at(bv[ks & 1][b / RY], b % RY),
                                                FIRST && ks == 0 ? accv{} : acc[a][b]);
                // interleave: each of the next step's LDS reads after a
                // share of this step's MFMAs
                if (ks + 1 < KT / 4) {
#pragma unroll
                    for (int r = 0; r < NREAD; ++r) {
                        __builtin_amdgcn_sched_group_barrier(0x008, NMFMA / NREAD, 0);
                        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
                    }
                }
            }
            return;
        }
        constexpr int UN = KU > 0 ? KU : KT / 4;
#pragma unroll UN
        for (int ks = 0; ks < KT / 4; ++ks) {
            const int k = 4 * ks + g;
            typename XV::type av[RB / RX];
            typename YV::type bv[CB / RY];
#pragma unroll
            for (int gi = 0; gi < RB / RX; ++gi)
                av[gi] = *reinterpret_cast<const typename XV::type *>(xat(ks, k, gi));
#pragma unroll
            for (int gj = 0; gj < CB / RY; ++gj)
                bv[gj] = *reinterpret_cast<const typename YV::type *>(yat(ks, k, gj));
#pragma unroll
            for (int a = 0; a < RB; ++a)
#pragma unroll
                for (int b = 0; b < CB; ++b)
                    acc[a][b] = mfma16x16x4(XV::at(av[a / RX], a % RX), YV::at(bv[b / RY], b % RY),
                                            FIRST && ks == 0 ? accv{} : acc[a][b]);
        }
    }

    __device__ __forceinline__ void rows_of(const int *offCx, int grp, int *ox) const
    {
#pragma unroll
        for (int i = 0; i < RX; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r)
                ox[i * 4 + r] =
                    offCx[wm * WTM + block_row<RX>(grp * RX + i, Traits<T>::mrow(g, r))];
    }
    __device__ __forceinline__ void cols_vec(const int *offCy, int *oy) const
    {
#pragma unroll
        for (int cg = 0; cg < CGV; ++cg) oy[cg] = offCy[wn * WTN + cg * 16 * RY + RY * l16];
    }
    // tile-local first column of this lane's column group cg (vector C accesses)
    __device__ __forceinline__ int col_of(int cg) const { return wn * WTN + cg * 16 * RY + RY * l16; }
    // tile-local row of element q of row group grp of this lane
    __device__ __forceinline__ int row_of(int grp, int q) const
    {
        return wm * WTM + block_row<RX>(grp * RX + q / 4, Traits<T>::mrow(g, q % 4));
    }
    // column y lies in a run [kE, kE + E) wholly inside [y0, ylim)
    static __device__ __forceinline__ bool in_whole_run(int y, int y0, int ylim, int E)
    {
        const int k = y / E;
        return k * E >= y0 && (k + 1) * E <= ylim;
    }
    // alpha * acc of the column groups whose first column lies in [c0, c1)
    // into stage[row][col - c0] (row pitch `pitch`; vector C accesses only)
    __device__ __forceinline__ void stage(T *st, int pitch, int c0, int c1, T alpha) const
    {
        if constexpr (kVecC) {
#pragma unroll
            for (int grp = 0; grp < RB / RX; ++grp)
#pragma unroll
                for (int cg = 0; cg < CGV; ++cg) {
                    const int col = col_of(cg);
                    if (col < c0 || col >= c1) continue;
#pragma unroll
                    for (int q = 0; q < NR; ++q) {
                        vec v;
#pragma unroll
                        for (int j = 0; j < VW; ++j) v[j] = alpha * acc[grp * RX + q / 4][cg * RY + j][q % 4];
                        *reinterpret_cast<vec *>(st + row_of(grp, q) * pitch + (col - c0)) = v;
                    }
                }
        }
    }

    // Unpack (Eq. 11): C <- alpha * acc + beta * C through C's offsets, RX
    // blocks of rows at a time (in PARTS parts of the rows, to bound the
    // registers held) -- every C load of a part first, so they are in flight
    // together, then the updates and non-temporal stores (C is written once
    // and not reused).  C is not read when beta == 0.
    //
    // E > 0 (vector C accesses only): skip the column groups that lie in a run
    // of E columns wholly inside the tile's columns [y0, ylim) -- those are
    // stored in C's memory order by unpack_c_order.
    //
    // ALL: every row and column of the tile lies inside C (no offset checks,
    // so every wavefront issues every store).
    template <int PARTS = 1, bool ALL = false>
    __device__ __forceinline__ void unpack(T *__restrict__ C, const int *offCx, const int *offCy,
                                           T alpha, T beta, bool cvec, int y0 = 0, int ylim = 0,
                                           int E = 0) const
    {
        static_assert(NR % PARTS == 0, "row parts");
        constexpr int NP = NR / PARTS;
        const bool readC = beta != T(0);
#pragma unroll
        for (int grp = 0; grp < RB / RX; ++grp) {
            int ox[NR];
            rows_of(offCx, grp, ox);
            if (kVecC && cvec) {
                int oy[CGV];
                cols_vec(offCy, oy);
                if (E > 0) {
#pragma unroll
                    for (int cg = 0; cg < CGV; ++cg)
                        if (in_whole_run(y0 + col_of(cg), y0, ylim, E)) oy[cg] = -1;
                }
#pragma unroll
                for (int part = 0; part < PARTS; ++part) {
                    vec cv[NP][CGV];
                    if (readC) {
#pragma unroll
                        for (int p = 0; p < NP; ++p)
#pragma unroll
                            for (int cg = 0; cg < CGV; ++cg)
                                if (ALL || (ox[part * NP + p] >= 0 && oy[cg] >= 0))
                                    cv[p][cg] = __builtin_nontemporal_load(reinterpret_cast<const vec *>(
                                        C + ox[part * NP + p] + oy[cg]));
                    }
#pragma unroll
                    for (int p = 0; p < NP; ++p)
#pragma unroll
                        for (int cg = 0; cg < CGV; ++cg) {
                            const int q = part * NP + p;
                            if (!ALL && (ox[q] < 0 || oy[cg] < 0)) continue;
                            vec out;
#pragma unroll
                            for (int j = 0; j < VW; ++j) {
                                const T a =
                                    alpha * acc[grp * RX + q / 4][kVecC ? cg * RY + j : 0][q % 4];
                                out[j] = readC ? a + beta * cv[p][cg][j] : a;
                            }
                            __builtin_nontemporal_store(out,
                                                        reinterpret_cast<vec *>(C + ox[q] + oy[cg]));
                        }
                }
            } else {
                int oy[CB];
#pragma unroll
                for (int b = 0; b < CB; ++b) oy[b] = offCy[wn * WTN + block_row<RY>(b, l16)];
#pragma unroll
                for (int part = 0; part < PARTS; ++part) {
                    T cv[NP][CB];
                    if (readC) {
#pragma unroll
                        for (int p = 0; p < NP; ++p)
#pragma unroll
                            for (int b = 0; b < CB; ++b)
                                if (ALL || (ox[part * NP + p] >= 0 && oy[b] >= 0))
                                    cv[p][b] = __builtin_nontemporal_load(C + ox[part * NP + p] + oy[b]);
                    }
#pragma unroll
                    for (int p = 0; p < NP; ++p)
#pragma unroll
                        for (int b = 0; b < CB; ++b) {
                            const int q = part * NP + p;
                            if (!ALL && (ox[q] < 0 || oy[b] < 0)) continue;
                            const T a = alpha * acc[grp * RX + q / 4][b][q % 4];
                            __builtin_nontemporal_store(readC ? a + beta * cv[p][b] : a,
                                                        C + ox[q] + oy[b]);
                        }
                }
            }
        }
    }

    // A partial tile (one piece of a tile's K boxes) in the workspace, in
    // lane order: element r of accumulator (a, b) of thread tid at
    // (((a CB + b) 4 + r) NTH + tid), so each store or load instruction of a
    // wavefront covers 64 consecutive elements and any workgroup of the same
    // kernel reads its own registers' values back.  Written and read with
    // device-scope accesses (relaxed atomics at agent scope): they bypass the
    // L2 of the XCD, which other XCDs do not see, so no cache-wide write-back
    // or invalidation (a fence) is needed between workgroups.
    template <int NTH>
    __device__ __forceinline__ void save(T *__restrict__ slot, int tid) const
    {
#pragma unroll
        for (int a = 0; a < RB; ++a)
#pragma unroll
            for (int b = 0; b < CB; ++b)
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    __hip_atomic_store(slot + (size_t)(((a * CB + b) * 4 + r) * NTH + tid),
                                       acc[a][b][r], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    // acc <- sum of the np saved pieces at slot0 + p * step (p = 0 .. np - 1,
    // added in that order), one row block at a time: the loads of a block
    // from up to NPB pieces are issued together (the reads come from device
    // memory; one round trip per block and group of pieces), and no more
    // than that are in flight (all of them would take more registers than
    // the accumulators).
    template <int NTH>
    __device__ __forceinline__ void sum_saved(const T *__restrict__ slot0, size_t step, int np,
                                              int tid)
    {
        constexpr int NPB = 2;
#pragma unroll
        for (int a = 0; a < RB; ++a) {
            for (int p0 = 0; p0 < np; p0 += NPB) {
                T v[NPB][CB][4];
#pragma unroll
                for (int q = 0; q < NPB; ++q)
                    if (p0 + q < np) {
                        const T *slot = slot0 + (size_t)(p0 + q) * step;
#pragma unroll
                        for (int b = 0; b < CB; ++b)
#pragma unroll
                            for (int r = 0; r < 4; ++r)
                                v[q][b][r] = __hip_atomic_load(
                                    slot + (size_t)(((a * CB + b) * 4 + r) * NTH + tid),
                                    __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    }
#pragma unroll
                for (int q = 0; q < NPB; ++q)
                    if (p0 + q < np) {
#pragma unroll
                        for (int b = 0; b < CB; ++b)
#pragma unroll
                            for (int r = 0; r < 4; ++r)
                                acc[a][b][r] = p0 + q == 0 ? v[q][b][r] : acc[a][b][r] + v[q][b][r];
                    }
            }
            __builtin_amdgcn_sched_barrier(0);
        }
    }
};

// ---------------------------------------------------------------------------
// Unpack in C's memory order, for a C whose stride-one run (E elements of the
// first column index) is shorter than a cache line while the next index in
// memory is a row index: the per-lane stores of the MFMA layout would write
// each 16-lane piece of a row into several runs, partial lines all.  The
// columns of every run wholly inside the tile are staged in LDS (the packing
// buffers, free after the K loop; as many runs per pass as fit in `cap`
// elements) and the workgroup stores them as (run, row, 16-byte piece) in
// order, so consecutive lanes write consecutive addresses through a run and
// on across rows.  Columns of runs cut by the tile's edges are stored per lane.
template <typename T, int MT, int NTH, typename WT>
__device__ __forceinline__ void unpack_c_order(const WT &w, T *__restrict__ C, T *stage, int cap,
                                               const int *offCx, const int *offCy, int y0,
                                               int ylim, int E, T alpha, T beta, int tid)
{
    constexpr int VW = Traits<T>::VW;
    typedef typename Traits<T>::vec vec;
    w.unpack(C, offCx, offCy, alpha, beta, true, y0, ylim, E);   // runs cut by the edges
    const int k0 = (y0 + E - 1) / E, k1 = ylim / E;            // whole runs [k0, k1)
    if (k1 <= k0) return;
    const int perPass = (cap / MT - VW) / E;                   // >= 1 (checked by the plan)
    const int pitch = perPass * E + VW;
    const int pieces = E / VW;                                 // 16-byte pieces per run row
    const bool readC = beta != T(0);
    for (int ka = k0; ka < k1; ka += perPass) {
        const int kb = min(k1, ka + perPass);
        const int c0 = ka * E - y0, c1 = kb * E - y0;         // tile-local columns of the pass
        __syncthreads();   // the LDS is free: the last MFMAs or the previous pass are done
        w.stage(stage, pitch, c0, c1, alpha);
        __syncthreads();
        const int n = (kb - ka) * MT * pieces;
        for (int L = tid; L < n; L += NTH) {
            const int run = L / (MT * pieces);
            const int rest = L - run * (MT * pieces);
            const int row = rest / pieces;
            const int col = c0 + run * E + (rest - row * pieces) * VW;
            const int ox = offCx[row];
            if (ox < 0) continue;   // a row outside the tensor
            vec v = *reinterpret_cast<const vec *>(stage + row * pitch + (col - c0));
            T *dst = C + ox + offCy[col];
            if (readC) {
                const vec c = __builtin_nontemporal_load(reinterpret_cast<const vec *>(dst));
#pragma unroll
                for (int j = 0; j < VW; ++j) v[j] += beta * c[j];
            }
            __builtin_nontemporal_store(v, reinterpret_cast<vec *>(dst));
        }
    }
}

// ---------------------------------------------------------------------------
// How a piece of work ends: the whole tile stored with alpha / beta, or a
// partial tile saved to workspace slot `slot`, the last of the tile's `np`
// pieces to arrive (counter `ctr`) summing slots base + p * step,
// p = 0 .. np - 1, in that order and storing the tile.
struct Part {
    enum { kWhole = 0, kSaved = 1 };
    int how = kWhole;
    int np = 1, slot = 0, base = 0, step = 1, ctr = 0;
};

// ---------------------------------------------------------------------------
// The macro-kernel: one tile per workgroup, any number of K boxes, NBUF LDS
// buffers (one suits a contracted set that fits one box).  With PF = 1 the gathers of box s+1 are issued before the MFMAs
// of box s; with PF = 2 there are two register stages and the gathers of box
// s+2 are issued before the MFMAs of box s, so a gather has two boxes' worth
// of MFMA time to arrive before its values are written to LDS.
//
// Kernel variants: whole tiles (SLICED = TAIL = 0: one tile per workgroup,
// from tile tile0 on), K slices (SLICED = 1) and the stream-K tail (TAIL = 1);
// only the last two carry the partial-tile code (its registers would cost the
// plain kernel occupancy or spills).
template <typename T, int MT, int NT, int KT, int WM, int WN, int RX, int RY, int WPE, int PF,
          int NBUF, int XMODE, int YMODE, int ONEBOX = 0, int CORDER = 0, int TAIL = 0,
          int SLICED = 0>
__global__ void __launch_bounds__(WM *WN * 64) __attribute__((amdgpu_waves_per_eu(WPE)))
gett_macro_kernel(const KDesc d, const T *__restrict__ X, const T *__restrict__ Y,
                  T *__restrict__ C, const T alpha, const T beta, T *__restrict__ W,
                  int *__restrict__ cnt)
{
    static_assert(PF == 1 || PF == 2, "prefetch depth");
    static_assert(NBUF == 2 || (NBUF == 1 && PF == 1), "one LDS buffer goes with one stage");
    static_assert(!ONEBOX || (NBUF == 1 && PF == 1), "the one-box kernel has one stage");
    static_assert(!(TAIL && SLICED), "one variant at a time");
    constexpr bool kPartials = TAIL || SLICED;
    constexpr int NTH = WM * WN * 64;
    // the k-vector swizzle only beside a vector gather of the other operand
    typedef Gather<T, MT, KT, XMODE, NTH, PF, YMODE == kGatherRowVec || YMODE == kGatherKVec> GX;
    typedef Gather<T, NT, KT, YMODE, NTH, PF, XMODE == kGatherRowVec || XMODE == kGatherKVec> GY;
    typedef WaveTile<T, MT, NT, KT, WM, WN, RX, RY> WT;

    // the packed panels; after the K loop the same memory stages C for
    // unpack_c_order
    constexpr int kPanels = NBUF * KT * (GX::PITCH + GY::PITCH);
    __shared__ __attribute__((aligned(16))) T panels[kPanels];
    T(*xs)[KT * GX::PITCH] = reinterpret_cast<T(*)[KT * GX::PITCH]>(panels);
    T(*ys)[KT * GY::PITCH] = reinterpret_cast<T(*)[KT * GY::PITCH]>(panels + NBUF * KT * GX::PITCH);
    // Offsets relative to the tile's base offsets (TileBase) and to the box
    // origin fit in 31 bits (the plan checks the spans); -1 marks a row or
    // column outside the tensor.
    __shared__ int rowX[MT], rowY[NT], offCx[MT], offCy[NT];
    __shared__ int kX[KT], kY[KT];
    __shared__ int kco[KT];
    __shared__ int permX[XMODE == kGatherScalar ? MT : 1], permY[YMODE == kGatherScalar ? NT : 1];
    __shared__ int lastPiece;   // this workgroup holds the last piece of its tile to arrive
    __shared__ int zeroLds;     // 0 (see the stream-K tail)

    const int tid = (int)threadIdx.x;
    const int ntiles = d.tilesX * d.tilesY;
    box_tables<KT, NTH>(d, tid, kX, kY, kco);
    WT w;

    // One piece of work: boxes [s0, s0 + nsteps) of the contracted set for
    // tile `tile` (a tile id in the order tile_of_block deals them), finished
    // as `part` says: the whole tile stored with alpha / beta, or a partial
    // tile summed in a fixed order through the workspace.  `tid` is the
    // thread index (passed in: see the stream-K tail).
    auto piece = [&](int tile, uint32_t s0, uint32_t nsteps, const Part &part, int tid) {
        w.init(tid);
        int tx, ty;
        tile_of_block(d, tile, ntiles, tx, ty);
        const TileBase tb = tile_base<MT, NT>(d, tx, ty);
        tile_tables<MT, NT, NTH>(d, tx, ty, tb, tid, rowX, offCx, rowY, offCy);
        const T *Xt = X + tb.x;
        const T *Yt = Y + tb.y;
        T *Ct = C + (tb.cx + tb.cy);
        if (XMODE == kGatherScalar && d.xperm > 0) row_perm<MT, NTH>(d.xperm, tx * MT, tid, permX);
        if (YMODE == kGatherScalar && d.yperm > 0) row_perm<NT, NTH>(d.yperm, ty * NT, tid, permY);
        __syncthreads();

        GX gx;
        GY gy;
        gx.setup(tid, rowX, kX, kco, d.xscalar_kfast, 1,
                 XMODE == kGatherScalar && d.xperm > 0 ? permX : nullptr);
        gy.setup(tid, rowY, kY, kco, d.yscalar_kfast, d.yes,
                 YMODE == kGatherScalar && d.yperm > 0 ? permY : nullptr);
        if (!ONEBOX) w.zero();
        BoxWalker walk;
        if constexpr (!ONEBOX) {
            if (nsteps > 0) walk.init(d, s0);   // fetch runs only when there are boxes
        }
        auto fetch = [&](auto stage, uint32_t s) {
            constexpr int B = decltype(stage)::value;
            int64_t ox, oy;
            const int lim = walk.at(d, s0 + s, ox, oy);
            gx.template load<B>(Xt + ox, lim);
            gy.template load<B>(Yt + oy, lim);
        };
        typedef std::integral_constant<int, 0> S0;
        typedef std::integral_constant<int, 1> S1;
        if constexpr (ONEBOX) {
            // Gather and pack X, then Y, then multiply: nothing in flight across
            // the MFMAs, one operand's values staged at a time, and the
            // accumulators first written by the MFMAs (a contracted set in one
            // box needs no more).  Plans with more boxes (a tile forced onto
            // them) take the same steps box after box, copying item by item.
            if (nsteps == 1) {
                int64_t ox, oy;
                const int lim = box_origin(d, s0, ox, oy);
                gx.template load<0>(Xt + ox, lim);
                gx.template store<0>(xs[0]);
                gy.template load<0>(Yt + oy, lim);
                gy.template store<0>(ys[0]);
                __syncthreads();
                w.template macro<GX::PITCH, GY::PITCH, true, 2, false, GX::kSwz, GY::kSwz>(xs[0], ys[0]);
            } else {
                w.zero();
                for (uint32_t s = 0; s < nsteps; ++s) {
                    int64_t ox, oy;
                    const int lim = box_origin(d, s0 + s, ox, oy);
                    if (s > 0) __syncthreads();   // the MFMAs of the previous box are done
                    gx.copy(Xt + ox, lim, xs[0]);
                    gy.copy(Yt + oy, lim, ys[0]);
                    __syncthreads();
                    w.template macro<GX::PITCH, GY::PITCH, false, 2, false, GX::kSwz, GY::kSwz>(xs[0], ys[0]);
                }
            }
        } else if constexpr (PF == 1) {
            if (nsteps > 0) {
                fetch(S0(), 0);
                gx.template store<0>(xs[0]);
                gy.template store<0>(ys[0]);
            }
            __syncthreads();
            for (uint32_t s = 0; s < nsteps; ++s) {
                const int buf = NBUF == 2 ? (int)(s & 1) : 0;
                const bool more = s + 1 < nsteps;
                if (more) fetch(S0(), s + 1);
                // one wavefront per SIMD over 4-step boxes: reads interleaved
                // with the MFMAs (measured faster there, not for 8-step boxes)
                w.template macro<GX::PITCH, GY::PITCH, false, 0, WPE == 1 && KT == 16, GX::kSwz,
                                 GY::kSwz>(xs[buf], ys[buf]);
                if (NBUF == 1 && more) __syncthreads();   // the single buffer is free again
                if (more) {
                    gx.template store<0>(xs[NBUF == 2 ? buf ^ 1 : 0]);
                    gy.template store<0>(ys[NBUF == 2 ? buf ^ 1 : 0]);
                }
                __syncthreads();
            }
        } else {
            // One box: start the gathers of box s+2 into this stage's registers,
            // run the MFMAs of box s from LDS buffer B, move box s+1's registers
            // into the other buffer.
            auto step = [&](auto stage, uint32_t s) {
                constexpr int B = decltype(stage)::value;
                if (s + 2 < nsteps) fetch(stage, s + 2);
                w.template macro<GX::PITCH, GY::PITCH, false, 0, false, GX::kSwz, GY::kSwz>(
                    xs[B % NBUF], ys[B % NBUF]);
                if (s + 1 < nsteps) {
                    gx.template store<B ^ 1>(xs[(B ^ 1) % NBUF]);
                    gy.template store<B ^ 1>(ys[(B ^ 1) % NBUF]);
                }
                __syncthreads();
            };
            if (nsteps > 0) {
                fetch(S0(), 0);
                if (nsteps > 1) fetch(S1(), 1);
                gx.template store<0>(xs[0]);
                gy.template store<0>(ys[0]);
            }
            __syncthreads();
            for (uint32_t s = 0; s < nsteps; s += 2) {
                step(S0(), s);
                if (s + 1 < nsteps) step(S1(), s + 1);
            }
        }
        if constexpr (kPartials) {
        if (part.how == Part::kSaved) {
            // Save this piece, count it; the last of the tile's pieces to
            // arrive sums all of them in piece order (a sum that does not
            // depend on which workgroup finished when) and stores the tile.
            // The saved values are written device-wide; each wavefront waits
            // until its stores have completed (vmcnt 0) before the barrier, so
            // the count that follows it comes after all of them, and the last
            // piece's device-wide reads come after the count.
            w.template save<NTH>(W + (size_t)part.slot * (MT * NT), tid);
            __builtin_amdgcn_s_waitcnt(kWaitStores);
            __syncthreads();
            if (tid == 0)
                lastPiece = __hip_atomic_fetch_add(cnt + part.ctr, 1, __ATOMIC_RELAXED,
                                                   __HIP_MEMORY_SCOPE_AGENT) == part.np - 1;
            __syncthreads();
            if (!lastPiece) return;
            w.template sum_saved<NTH>(W + (size_t)part.base * (MT * NT),
                                      (size_t)part.step * (MT * NT), part.np, tid);
            if (tid == 0)   // zero again for the next call
                __hip_atomic_store(cnt + part.ctr, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        }
        if constexpr (CORDER && WT::kVecC) {   // compiled only into the tiles that carry it
            if (d.crun > 0 && d.cvec) {
                const int y0 = ty * NT;
                const int ylim = (int)min((int64_t)y0 + NT, d.sizeY);
                unpack_c_order<T, MT, NTH>(w, Ct, panels, kPanels, offCx, offCy, y0, ylim, d.crun,
                                           alpha, beta, tid);
                return;
            }
        }
        w.template unpack<ONEBOX ? 2 : 1>(Ct, offCx, offCy, alpha, beta, d.cvec != 0);
    };

    if constexpr (TAIL) {
        // Stream-K tail: workgroups below tailFull compute one whole tile
        // each; every later one sums a run of tailLen consecutive boxes of the
        // concatenated box sequences of the remaining tiles (the end of one
        // tile and the start of the next, possibly).  A run that holds a tail
        // tile whole stores it; the pieces of a tile shared by several runs
        // are summed through the workspace.  Piece p of tail tile u comes from
        // run jf(u) + p, jf(u) = floor(u nb / tailLen), and is saved in slot
        // jf(u) + p + u: slots grow with (u, p), so they are distinct.
        //
        // Both kinds of workgroup walk one loop (one copy of the piece code):
        // positions are boxes of the concatenated sequences of all tiles; a
        // whole-tile workgroup's run is its tile.  The thread index each
        // piece sees is read through LDS, so the compiler keeps nothing
        // derived from it alive from one piece to the next (across the K
        // loop, where registers are short).
        if (tid == 0) zeroLds = 0;
        __syncthreads();
        const int bid = (int)blockIdx.x;
        const uint64_t nb = (uint64_t)d.nsteps;
        const uint64_t L = (uint64_t)d.tailLen;
        const uint64_t first = (uint64_t)d.tailFull * nb;   // first box of the tail tiles
        const int j = bid - d.tailFull;                      // tail run (j >= 0)
        uint64_t pos = j < 0 ? (uint64_t)bid * nb : first + (uint64_t)j * L;
        const uint64_t end = j < 0 ? pos + nb : min(pos + L, (uint64_t)ntiles * nb);
        while (pos < end) {
            const uint64_t t = pos / nb;
            const uint32_t s0 = (uint32_t)(pos - t * nb);
            const uint32_t n = (uint32_t)min(nb - s0, end - pos);
            const uint64_t u = t - (uint64_t)d.tailFull;   // tail tile (when j >= 0)
            Part part;
            if (j >= 0 && n < nb) {
                const int jf = (int)(u * nb / L);
                const int jl = (int)(((u + 1) * nb - 1) / L);
                part.how = Part::kSaved;
                part.np = jl - jf + 1;
                part.slot = j + (int)u;
                part.base = jf + (int)u;
                part.step = 1;
                part.ctr = (int)u;
            }
            piece((int)t, s0, n, part, tid + *reinterpret_cast<volatile int *>(&zeroLds));
            pos += n;
            if (pos < end) __syncthreads();   // the next piece rewrites the tables and panels
        }
    } else if constexpr (!SLICED) {
        // whole tiles: workgroup b computes tile tile0 + b (tile0 > 0 for a
        // pass that scales the tail tiles of a stream-K plan)
        piece(d.tile0 + (int)blockIdx.x, 0, (uint32_t)d.nsteps, Part{}, tid);
    } else {
        // K slices: workgroup b computes slice b / tiles of tile b % tiles.
        // Slice p of tile u is saved in slot p * tiles + u.
        const int slices = d.kslices > 1 ? d.kslices : 1;
        const int span = ntiles - d.tile0;
        const int bid = (int)blockIdx.x;
        const int slice = slices > 1 ? bid / span : 0;
        const uint32_t s0 = (uint32_t)((uint64_t)d.nsteps * slice / slices);
        const uint32_t n = (uint32_t)((uint64_t)d.nsteps * (slice + 1) / slices) - s0;
        const int u = bid - slice * span;
        Part part;
        if (slices > 1) {
            part.how = Part::kSaved;
            part.np = slices;
            part.slot = slice * span + u;
            part.base = u;
            part.step = span;
            part.ctr = u;
        }
        piece(d.tile0 + u, s0, n, part, tid);
    }
}

// ---------------------------------------------------------------------------
// The streaming kernel, for contractions whose contracted set fits in one K
// box (the panel-panel case of Table I: k small) and whose time goes to the C
// stream.  A persistent workgroup walks tiles t = blockIdx.x, + gridDim.x, ...
// in C's memory order (y fastest), so the workgroups running together write
// neighbouring stretches of C, and overlaps each tile's stores with the next
// tile's packing and MFMAs.  With tile t's results in the accumulators:
//   tables(t+1); barrier; issue the gathers of t+1; unpack(t);
//   store the gathered panels of t+1 to LDS; barrier; macro(t+1).
// A wavefront's vector memory operations count down in the order they were
// issued, so waiting for the gathers of t+1 -- issued before the stores of
// t -- does not wait for those stores: they drain behind the packing and
// the MFMAs of t+1.
template <typename T, int MT, int NT, int KT, int WM, int WN, int RX, int RY, int WPE, int XMODE,
          int YMODE>
__global__ void __launch_bounds__(WM *WN * 64) __attribute__((amdgpu_waves_per_eu(WPE)))
gett_stream_kernel(const KDesc d, const T *__restrict__ X, const T *__restrict__ Y,
                   T *__restrict__ C, const T alpha, const T beta)
{
    constexpr int NTH = WM * WN * 64;
    typedef Gather<T, MT, KT, XMODE, NTH, 1, YMODE == kGatherRowVec || YMODE == kGatherKVec> GX;
    typedef Gather<T, NT, KT, YMODE, NTH, 1, XMODE == kGatherRowVec || XMODE == kGatherKVec> GY;
    typedef WaveTile<T, MT, NT, KT, WM, WN, RX, RY> WT;

    __shared__ __attribute__((aligned(16))) T xs[KT * GX::PITCH];
    __shared__ __attribute__((aligned(16))) T ys[KT * GY::PITCH];
    __shared__ int rowX[2][MT], rowY[2][NT], offCx[2][MT], offCy[2][NT];
    __shared__ int kX[KT], kY[KT];
    __shared__ int kco[KT];

    const int tid = (int)threadIdx.x;
    const int ntiles = d.tilesX * d.tilesY;
    const int G = (int)gridDim.x;
    int t = (int)blockIdx.x;
    if (t >= ntiles) return;   // uniform per workgroup; the host never launches more

    const bool withK = d.nsteps > 0;   // 0: alpha == 0 or an empty sum, A and B unread
    int64_t ox0 = 0, oy0 = 0;
    int lim = 0;
    if (withK) lim = box_origin(d, 0, ox0, oy0);

    box_tables<KT, NTH>(d, tid, kX, kY, kco);
    TileBase cb = tile_base<MT, NT>(d, t / d.tilesY, t % d.tilesY);
    tile_tables<MT, NT, NTH>(d, t / d.tilesY, t % d.tilesY, cb, tid, rowX[0], offCx[0], rowY[0],
                             offCy[0]);
    __syncthreads();

    GX gx;
    GY gy;
    WT w;
    w.init(tid);
    w.zero();
    if (withK) {
        gx.setup(tid, rowX[0], kX, kco, d.xscalar_kfast);
        gy.setup(tid, rowY[0], kY, kco, d.yscalar_kfast, d.yes);
        gx.load(X + (cb.x + ox0), lim);
        gy.load(Y + (cb.y + oy0), lim);
        gx.store(xs);
        gy.store(ys);
        __syncthreads();
        w.template macro<GX::PITCH, GY::PITCH, true, 0, false, GX::kSwz, GY::kSwz>(xs, ys);
    }

    for (int j = 0; t < ntiles; ++j, t += G) {
        const int cur = j & 1;
        const int tn = t + G;
        const bool more = tn < ntiles;
        TileBase nb = cb;
        // the tables of t+1 go to the other set: tile t's gathers took theirs
        // into registers, and tile t-1's stores have their addresses
        if (more) {
            nb = tile_base<MT, NT>(d, tn / d.tilesY, tn % d.tilesY);
            tile_tables<MT, NT, NTH>(d, tn / d.tilesY, tn % d.tilesY, nb, tid, rowX[cur ^ 1],
                                     offCx[cur ^ 1], rowY[cur ^ 1], offCy[cur ^ 1]);
        }
        __syncthreads();   // tables of t+1 written; every wavefront's MFMAs of t read the panels
        if (more && withK) {
            gx.setup(tid, rowX[cur ^ 1], kX, kco, d.xscalar_kfast);
            gy.setup(tid, rowY[cur ^ 1], kY, kco, d.yscalar_kfast, d.yes);
            gx.load(X + (nb.x + ox0), lim);
            gy.load(Y + (nb.y + oy0), lim);
        }
        w.template unpack<2>(C + (cb.cx + cb.cy), offCx[cur], offCy[cur], alpha, beta, d.cvec != 0);
        cb = nb;
        if (!more) break;
        if (withK) {
            gx.store(xs);
            gy.store(ys);
        }
        __syncthreads();   // panels of t+1 written
        if (withK) w.template macro<GX::PITCH, GY::PITCH, true, 0, false, GX::kSwz, GY::kSwz>(xs, ys);
        else w.zero();
    }
}

}  // namespace gett
