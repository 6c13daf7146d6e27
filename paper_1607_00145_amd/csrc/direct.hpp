// direct.hpp -- the direct-load variants of the macro-kernel (device code).
//
// When both operands are gathered in 16-byte vectors (row or k vectors),
// packing (Eq. 9-10) needs no registers: the load unit copies each 16-byte
// piece from device memory straight into LDS (global_load_lds_dwordx4: lane
// i of one instruction fills bytes [16 i, 16 i + 16) after a wave-uniform LDS
// base); a piece outside the tensors is written as zeros by its thread.
// The LDS layout of an operand tile is then fixed by which piece each lane
// loads:
//   row-vector operand: [k][row], as the macro-kernel packs it (no padding);
//   k-vector operand:   [row][k], the pieces of row r XOR-permuted by
//                       (r / R) mod (pieces per row) -- rotated by r / R when
//                       the pieces per row are not a power of two -- so that
//                       the lanes of an MFMA read, which take rows R apart at
//                       one k piece (R = 4 in fp32, 2 in fp64), fall on
//                       different banks.
// A k-vector piece holds VW consecutive contracted positions, and one LDS
// read hands them to VW consecutive MFMA steps: the position lane group g
// supplies in step s is
//   kp(s, g) = 4 VW floor(s / VW) + VW g + (s mod VW)
// on both operands (a bijection of the box's KT positions onto the (s, g)
// pairs, so each product still pairs matching indices and the sum is the
// same up to rounding order).
//
// Pipeline, two LDS buffers, box s in buffer s mod 2:
//   MFMAs of box s's first step groups, from registers;
//   wait for this wavefront's loads of box s + 1; barrier (all loads of box
//     s + 1 have landed, every wavefront is done reading box s);
//   loads of box s + 2 into box s's buffer;
//   LDS reads of box s + 1's fragments, interleaved with the MFMAs of box s's
//     last step group.
// Nothing is staged in registers but the fragments, so a workgroup of eight
// wavefronts (two per SIMD) fits a 256 x 128 fp32 tile.
//
// The persistent variant (gett_direct_stream_kernel, contracted sets of one
// box) walks several tiles per workgroup and copies the next tile's box into
// the other buffer before storing the current tile's C, so the copy is not
// queued behind those stores.
#pragma once
#include "kernel.hpp"

namespace gett {

typedef __attribute__((address_space(1))) void global_void;
typedef __attribute__((address_space(3))) void lds_void;

// k-vector layout: LDS column of piece c of row r (CPR pieces per row, rows
// read R at a time).  With 2^n pieces per row the pieces are XOR-permuted by
// (r / R) mod CPR (an involution); otherwise rotated by r / R.
template <int CPR, int R>
__device__ __forceinline__ int kvec_col(int r, int c)
{
    if constexpr ((CPR & (CPR - 1)) == 0) return c ^ ((r / R) & (CPR - 1));
    else return (c + r / R) % CPR;
}
// the piece of row r held in LDS column c
template <int CPR, int R>
__device__ __forceinline__ int kvec_piece(int r, int c)
{
    if constexpr ((CPR & (CPR - 1)) == 0) return c ^ ((r / R) & (CPR - 1));
    else return (c + CPR - (r / R) % CPR) % CPR;
}

// The pieces of one operand tile (ROWS x KT elements) one thread loads per
// box: J per thread, piece p = (j * NW + wave) * 64 + lane of the tile's LDS
// image.  A piece outside the tensor (its rows past the tile's last, or its
// contracted positions past the box's valid ones) is not loaded: the thread
// writes zeros to its place instead, as the macro-kernel's gathers do.
// WHOLE: every piece of every box is inside (no checks).  R: rows one lane
// reads together from the [row][k] layout (RX / RY), which sets the row
// period of the k-vector permutation.
template <typename T, int ROWS, int KT, int MODE, int NTH, bool WHOLE, int R>
struct DirectOperand {
    static constexpr int VW = Traits<T>::VW;
    static constexpr int NW = NTH / 64;
    static constexpr int PIECES = ROWS * KT / VW;
    static constexpr int J = PIECES / NTH;
    static constexpr int CPR = KT / VW;     // k-vector layout: pieces per row
    static constexpr int RPL = ROWS / VW;   // row-vector layout: pieces per line
    static_assert(MODE == kGatherRowVec || MODE == kGatherKVec, "vector gathers only");
    static_assert(PIECES % NTH == 0 && J >= 1, "whole pieces per thread");
    static_assert(ROWS % VW == 0 && KT % VW == 0, "whole vectors");
    typedef typename Traits<T>::vec vec;

    int goff[J];               // element offset of each piece (tile base and box origin excluded)
    int kc[WHOLE ? 1 : J];     // position along index kj of its first element; kInvalidK: never valid
    int lane;

    // piece of row r held in LDS column c of the k-vector layout (the inverse
    // of kvec_col)
    static __device__ __forceinline__ int swz(int r, int c) { return kvec_piece<CPR, R>(r, c); }

    // rowoff: LDS table of operand offsets per tile row (-1 = outside the
    // tensor); koff / kco: offsets / kj-positions per box position
    __device__ __forceinline__ void setup(int tid, const int *rowoff, const int *koff,
                                          const int *kco)
    {
        lane = tid & 63;
        const int w = tid >> 6;
#pragma unroll
        for (int j = 0; j < J; ++j) {
            const int p = (j * NW + w) * 64 + lane;
            int r, kk;
            if constexpr (MODE == kGatherKVec) {
                r = p / CPR;
                kk = VW * swz(r, p % CPR);
            } else {
                r = VW * (p % RPL);
                kk = p / RPL;
            }
            const int ro = rowoff[r];
            goff[j] = (ro < 0 ? 0 : ro) + koff[kk];
            if constexpr (!WHOLE) kc[j] = ro < 0 ? kInvalidK : kco[kk];
        }
    }

    // copy this thread's pieces of the box at `base` (`lim` valid positions
    // along index kj) into the tile image `dst`
    __device__ __forceinline__ void issue(const T *base, T *dst, int w, int lim) const
    {
#pragma unroll
        for (int j = 0; j < J; ++j) {
            T *slot = dst + (j * NW + w) * 64 * VW;
            if (WHOLE || kc[WHOLE ? 0 : j] < lim)
                __builtin_amdgcn_global_load_lds((global_void *)(base + goff[j]),
                                                 (lds_void *)slot, 16, 0, 0);
            else
                *reinterpret_cast<vec *>(slot + lane * VW) = vec{};
        }
    }
};

// Fragments of one step group (VW MFMA steps) for the NB blocks of one side
// of a wavefront's register tile.  Block b's lane l16 stands for tile row
// w0 + block_row<R>(b, l16), as in WaveTile.
template <typename T, int MODE, int NB, int R, int ROWS, int KT>
struct DirectFrag {
    static constexpr int VW = Traits<T>::VW;
    typedef typename Traits<T>::vec vec;
    typedef RVec<T, R> RV;
    static constexpr bool kKV = MODE == kGatherKVec;
    static constexpr int CPR = KT / VW;
    static constexpr int kReads = kKV ? NB : VW * (NB / R);   // LDS reads per group
    // k-vector: one piece per block (VW positions of its row); row-vector:
    // one read of R rows per block group for each of the VW steps
    vec kv[kKV ? NB : 1];
    typename RV::type rv[kKV ? 1 : VW][kKV ? 1 : NB / R];

    __device__ __forceinline__ void read(const T *tile, int w0, int l16, int g, int grp)
    {
        if constexpr (kKV) {
            const int q = 4 * grp + g;   // piece of positions kp(VW grp .. VW grp + VW - 1, g)
#pragma unroll
            for (int b = 0; b < NB; ++b) {
                const int r = w0 + block_row<R>(b, l16);
                kv[b] = *reinterpret_cast<const vec *>(tile + r * KT + VW * kvec_col<CPR, R>(r, q));
            }
        } else {
#pragma unroll
            for (int s4 = 0; s4 < VW; ++s4) {
                const int k = 4 * VW * grp + VW * g + s4;
#pragma unroll
                for (int gi = 0; gi < NB / R; ++gi)
                    rv[s4][gi] = *reinterpret_cast<const typename RV::type *>(
                        tile + k * ROWS + w0 + gi * 16 * R + R * l16);
            }
        }
    }
    // the value block b supplies in step s4 of the group
    __device__ __forceinline__ T at(int b, int s4) const
    {
        if constexpr (kKV) return kv[b][s4];
        else return RV::at(rv[s4][b / R], b % R);
    }
};

// Origins of the K boxes, taken in order (every box whole): the block along
// index kj advances by one; when it wraps, the next contracted index
// advances; only when that one wraps too is the origin decomposed afresh
// (box_origin).  The state is the same on every lane and is kept in scalar
// registers (as vector registers it cost the K loop 3% on the 4096^3-shaped
// fp32 contraction).
struct DirectWalk {
    int64_t ox, oy;     // origin of box `next` in X and Y
    int64_t bx, by;     // step of one block along index kj
    int64_t sx1, sy1;   // strides of index kj + 1
    uint32_t next;
    int blk, c1, nblk, e1, ek, tj;

    __device__ __forceinline__ void init(const KDesc &d)
    {
        nblk = d.nblk > 0 ? d.nblk : 1;
        ek = d.extK[d.kj];
        tj = d.tj;
        bx = (int64_t)d.tj * d.strXk[d.kj];
        by = (int64_t)d.tj * d.strYk[d.kj];
        const bool later = d.kj + 1 < d.nk;
        e1 = later ? d.extK[d.kj + 1] : 0;
        sx1 = later ? d.strXk[d.kj + 1] : 0;
        sy1 = later ? d.strYk[d.kj + 1] : 0;
        next = 0;
        blk = 0;
        c1 = 0;
        box_origin(d, 0, ox, oy);
    }
    // origin of box `next` and its valid positions along index kj; then step
    // to the box after it
    __device__ __forceinline__ int take(const KDesc &d, int64_t &x, int64_t &y)
    {
        x = ox;
        y = oy;
        const int lim = ek - blk * tj;
        ++next;
        if (++blk < nblk) {
            ox += bx;
            oy += by;
        } else if (++c1 < e1) {
            blk = 0;
            ox += sx1 - (int64_t)(nblk - 1) * bx;
            oy += sy1 - (int64_t)(nblk - 1) * by;
        } else {
            blk = 0;
            c1 = 0;
            box_origin(d, next, ox, oy);
        }
        blk = uniform(blk);
        c1 = uniform(c1);
        ox = uniform(ox);
        oy = uniform(oy);
        return lim;
    }
};

template <typename T, int MT, int NT, int KT, int WM, int WN, int RX, int RY, int XMODE,
          int YMODE, bool WHOLE>
__global__ void __launch_bounds__(WM *WN * 64) __attribute__((amdgpu_waves_per_eu(2)))
gett_direct_kernel(const KDesc d, const T *__restrict__ X, const T *__restrict__ Y,
                   T *__restrict__ C, const T alpha, const T beta)
{
    constexpr int NTH = WM * WN * 64;
    constexpr int VW = Traits<T>::VW;
    constexpr int NG = KT / (4 * VW);   // step groups per box
    static_assert(KT % (4 * VW) == 0, "whole step groups");
    typedef WaveTile<T, MT, NT, KT, WM, WN, RX, RY> WT;
    typedef DirectOperand<T, MT, KT, XMODE, NTH, WHOLE, RX> OX;
    typedef DirectOperand<T, NT, KT, YMODE, NTH, WHOLE, RY> OY;
    typedef DirectFrag<T, XMODE, WT::RB, RX, MT, KT> FX;
    typedef DirectFrag<T, YMODE, WT::CB, RY, NT, KT> FY;
    constexpr int STAGE = (MT + NT) * KT;

    // the two box buffers: dynamic LDS of 2 * STAGE elements (the compiler
    // then does not wait for the loads in flight into one buffer before
    // reading the other)
    extern __shared__ __attribute__((aligned(16))) char dyn_lds[];
    T *panels = reinterpret_cast<T *>(dyn_lds);
    __shared__ int rowX[MT], rowY[NT], offCx[MT], offCy[NT];
    __shared__ int kX[KT], kY[KT], kco[KT];

    const int tid = (int)threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int ntiles = d.tilesX * d.tilesY;
    box_tables<KT, NTH>(d, tid, kX, kY, kco);
    WT w;
    w.init(tid);
    int tx, ty;
    tile_of_block(d, d.tile0 + (int)blockIdx.x, ntiles, tx, ty);
    const TileBase tb = tile_base<MT, NT>(d, tx, ty);
    tile_tables<MT, NT, NTH>(d, tx, ty, tb, tid, rowX, offCx, rowY, offCy);
    const T *Xt = X + tb.x;
    const T *Yt = Y + tb.y;
    T *Ct = C + (tb.cx + tb.cy);
    __syncthreads();

    OX ox;
    OY oy;
    ox.setup(tid, rowX, kX, kco);
    oy.setup(tid, rowY, kY, kco);
    w.zero();
    const uint32_t nsteps = (uint32_t)d.nsteps;
    const int l16 = tid & 15, g = (tid & 63) >> 4;
    const int xw = w.wm * WT::WTM, yw = w.wn * WT::WTN;

    DirectWalk walk;
    if (nsteps > 0) walk.init(d);
    auto issue = [&](int buf) {   // the boxes in order: 0, 1, 2, ...
        int64_t bx, by;
        const int lim = walk.take(d, bx, by);
        T *st = panels + buf * STAGE;
        ox.issue(Xt + bx, st, wave, lim);
        oy.issue(Yt + by, st + MT * KT, wave, lim);
    };
    auto read = [&](FX (&fx)[NG], FY (&fy)[NG], int buf) {
        const T *st = panels + buf * STAGE;
#pragma unroll
        for (int grp = 0; grp < NG; ++grp) {
            fx[grp].read(st, xw, l16, g, grp);
            fy[grp].read(st + MT * KT, yw, l16, g, grp);
        }
    };
    auto mma = [&](const FX &fx, const FY &fy) {
#pragma unroll
        for (int s4 = 0; s4 < VW; ++s4)
#pragma unroll
            for (int a = 0; a < WT::RB; ++a)
#pragma unroll
                for (int b = 0; b < WT::CB; ++b)
                    w.acc[a][b] = mfma16x16x4(fx.at(a, s4), fy.at(b, s4), w.acc[a][b]);
    };
    // s_barrier with no fence: a workgroup-scope release would wait for the
    // loads in flight into the other buffer (they count as LDS writes)
    auto barrier = []() { asm volatile("s_barrier" ::: "memory"); };
    constexpr int LOADS = OX::J + OY::J;   // load instructions per box and thread
    // s_waitcnt: vmcnt n (gfx9 encoding: low bits 3:0, high bits 15:14),
    // expcnt and lgkmcnt untouched / lgkmcnt 0
    // (lgkmcnt 0 also covers the zeros written in place of pieces outside)
    constexpr int kVmBox = (LOADS & 15) | ((LOADS >> 4) << 14) | (7 << 4);
    constexpr int kVmLgk0 = 7 << 4;
    static_assert(LOADS < 64, "vmcnt range");

    if (nsteps > 0) {
        FX fx[NG];
        FY fy[NG];
        issue(0);
        if (nsteps > 1) {
            issue(1);
            // box 0's loads; box 1's may stay in flight when each box is known
            // to issue all of its loads (a wavefront skips the loads of
            // pieces that are all outside, so the count is not known otherwise)
            __builtin_amdgcn_s_waitcnt(WHOLE ? kVmBox : kVmLgk0);
        } else {
            __builtin_amdgcn_s_waitcnt(kVmLgk0);
        }
        barrier();
        read(fx, fy, 0);
        for (uint32_t s = 0; s + 1 < nsteps; ++s) {
#pragma unroll
            for (int grp = 0; grp + 1 < NG; ++grp) mma(fx[grp], fy[grp]);
            __builtin_amdgcn_s_waitcnt(kVmLgk0);   // box s + 1 loaded, box s read
            barrier();
            if (s + 2 < nsteps) issue((int)(s & 1));   // box s + 2
            FX gx[NG];
            FY gy[NG];
            read(gx, gy, (int)((s + 1) & 1));
            mma(fx[NG - 1], fy[NG - 1]);
            // one fragment read after every few MFMAs of the last group
            constexpr int NREAD = NG * (FX::kReads + FY::kReads);
            constexpr int NMFMA = VW * WT::RB * WT::CB;
#pragma unroll
            for (int r = 0; r < NREAD; ++r) {
                __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
                __builtin_amdgcn_sched_group_barrier(0x008, NMFMA / NREAD > 0 ? NMFMA / NREAD : 1,
                                                     0);
            }
#pragma unroll
            for (int grp = 0; grp < NG; ++grp) {
                fx[grp] = gx[grp];
                fy[grp] = gy[grp];
            }
        }
#pragma unroll
        for (int grp = 0; grp < NG; ++grp) mma(fx[grp], fy[grp]);
    }
    w.template unpack<1>(Ct, offCx, offCy, alpha, beta, d.cvec != 0);
}

// Persistent direct-load kernel for plans whose contracted set is one K box.
// Workgroups walk tiles t = tile0 + blockIdx.x, + gridDim.x, ...; tile t's box
// sits in LDS buffer t mod 2 (per workgroup).  Per tile:
//   LDS reads of tile t's fragments; offset tables of the next tile (second
//     table set); barrier;
//   the copy of the next tile's box into the other buffer;
//   MFMAs of tile t; its C stores (unpack);
//   wait for this wavefront's copy; barrier.
// The copy is issued before the C stores of tile t, so it does not queue
// behind them (a CU serves its vector memory instructions in order), and the
// wait for it leaves those stores in flight: vmcnt counts in issue order and
// every tile issues at least kStores vector memory instructions after its
// copy when every piece is inside the tensors (WHOLE); otherwise the wait
// is for everything (vmcnt 0).
template <typename T, int MT, int NT, int KT, int WM, int WN, int RX, int RY, int XMODE, int YMODE,
          bool WHOLE>
__global__ __launch_bounds__(WM * WN * 64) __attribute__((amdgpu_waves_per_eu(2))) void
gett_direct_stream_kernel(const KDesc d, const T *__restrict__ X, const T *__restrict__ Y,
                          T *__restrict__ C, const T alpha, const T beta)
{
    constexpr int NTH = WM * WN * 64;
    constexpr int VW = Traits<T>::VW;
    constexpr int NG = KT / (4 * VW);   // step groups per box
    static_assert(KT % (4 * VW) == 0, "whole step groups");
    typedef WaveTile<T, MT, NT, KT, WM, WN, RX, RY> WT;
    typedef DirectOperand<T, MT, KT, XMODE, NTH, WHOLE, RX> OX;
    typedef DirectOperand<T, NT, KT, YMODE, NTH, WHOLE, RY> OY;
    typedef DirectFrag<T, XMODE, WT::RB, RX, MT, KT> FX;
    typedef DirectFrag<T, YMODE, WT::CB, RY, NT, KT> FY;
    constexpr int STAGE = (MT + NT) * KT;
    // vector memory instructions each wavefront issues after a copy: the C
    // stores of one tile, vectors or single elements (C loads with beta != 0
    // only add to them)
    constexpr int kStores = (WT::RB / RX) * WT::NR * (WT::kVecC ? WT::CGV : WT::CB);
    constexpr int kAfter = kStores < 63 ? kStores : 63;
    // s_waitcnt (gfx9 encoding): vmcnt kAfter / vmcnt 0, lgkmcnt 0 / lgkmcnt
    // 0 alone (vmcnt 63), expcnt untouched
    constexpr int kVmAfter = (kAfter & 15) | ((kAfter >> 4) << 14) | (7 << 4) | (15 << 8);
    constexpr int kVmLgk0 = 7 << 4;
    constexpr int kLgk0 = 15 | (3 << 14) | (7 << 4);

    extern __shared__ __attribute__((aligned(16))) char dyn_lds[];
    T *panels = reinterpret_cast<T *>(dyn_lds);
    __shared__ int rowX[2][MT], rowY[2][NT], offCx[2][MT], offCy[2][NT];
    __shared__ int kX[KT], kY[KT], kco[KT];

    const int tid = (int)threadIdx.x;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int ntiles = d.tilesX * d.tilesY;
    box_tables<KT, NTH>(d, tid, kX, kY, kco);
    int64_t bx0, by0;
    const int lim = box_origin(d, 0, bx0, by0);
    WT w;
    w.init(tid);
    const int l16 = tid & 15, g = (tid & 63) >> 4;
    const int xw = w.wm * WT::WTM, yw = w.wn * WT::WTN;
    OX ox;
    OY oy;
    auto barrier = []() { asm volatile("s_barrier" ::: "memory"); };
    // offset tables of tile t into table set `set`; the tile's operand and C bases
    auto prepare = [&](int t, int set, const T *&Xt, const T *&Yt, T *&Ct) {
        int tx, ty;
        tile_of_block(d, t, ntiles, tx, ty);
        const TileBase tb = tile_base<MT, NT>(d, tx, ty);
        tile_tables<MT, NT, NTH>(d, tx, ty, tb, tid, rowX[set], offCx[set], rowY[set], offCy[set]);
        Xt = X + (tb.x + bx0);
        Yt = Y + (tb.y + by0);
        Ct = C + (tb.cx + tb.cy);
    };
    auto issue = [&](int set, const T *Xt, const T *Yt, int buf) {
        ox.setup(tid, rowX[set], kX, kco);
        oy.setup(tid, rowY[set], kY, kco);
        T *st = panels + buf * STAGE;
        ox.issue(Xt, st, wave, lim);
        oy.issue(Yt, st + MT * KT, wave, lim);
    };
    auto mma = [&](const FX &fx, const FY &fy) {
#pragma unroll
        for (int s4 = 0; s4 < VW; ++s4)
#pragma unroll
            for (int a = 0; a < WT::RB; ++a)
#pragma unroll
                for (int b = 0; b < WT::CB; ++b)
                    w.acc[a][b] = mfma16x16x4(fx.at(a, s4), fy.at(b, s4), w.acc[a][b]);
    };

    int t = d.tile0 + (int)blockIdx.x;   // the grid holds no more workgroups than tiles
    const T *Xt, *Yt;
    T *Ct;
    prepare(t, 0, Xt, Yt, Ct);
    __syncthreads();
    issue(0, Xt, Yt, 0);
    __builtin_amdgcn_s_waitcnt(kVmLgk0);
    barrier();
    int cur = 0;
    for (;;) {
        FX fx[NG];
        FY fy[NG];
        const T *st = panels + cur * STAGE;
#pragma unroll
        for (int grp = 0; grp < NG; ++grp) {
            fx[grp].read(st, xw, l16, g, grp);
            fy[grp].read(st + MT * KT, yw, l16, g, grp);
        }
        const int tn = t + (int)gridDim.x;
        const bool more = tn < ntiles;
        const T *Xn = Xt, *Yn = Yt;
        T *Cn = Ct;
        if (more) prepare(tn, cur ^ 1, Xn, Yn, Cn);
        // this tile's fragments are in registers, the next tile's tables complete
        __builtin_amdgcn_s_waitcnt(kLgk0);
        barrier();
        if (more) issue(cur ^ 1, Xn, Yn, cur ^ 1);
        // the copy stays ahead of the stores below in issue order
        __builtin_amdgcn_sched_barrier(0);
        asm volatile("" ::: "memory");
        w.zero();
#pragma unroll
        for (int grp = 0; grp < NG; ++grp) mma(fx[grp], fy[grp]);
        w.template unpack<1, WHOLE>(Ct, offCx[cur], offCy[cur], alpha, beta, d.cvec != 0);
        if (!more) break;
        __builtin_amdgcn_sched_barrier(0);
        asm volatile("" ::: "memory");
        // the next tile's box has landed (this wavefront's part; the barrier
        // covers the others); this tile's stores may still be in flight
        __builtin_amdgcn_s_waitcnt(WHOLE ? kVmAfter : kVmLgk0);
        barrier();
        t = tn;
        Xt = Xn;
        Yt = Yn;
        Ct = Cn;
        cur ^= 1;
    }
}

}  // namespace gett
