// desc.hpp -- plain-data kernel descriptor shared by the host analyser and
// the device kernels.
//
// The macro-kernel computes a tile of the matrix view C[x][y] of C, where
//   x runs over I_x, the free indices of the "row" operand X, and
//   y runs over I_y, the free indices of the "column" operand Y;
// (X, Y) is (A, B) or, when the operands are exchanged, (B, A).  Each free
// set is linearised in the analyser's order (first index fastest), which is
// how the paper's single m- and n-loops of Listing 4 stand for several
// indices each (Sec. 3, identify_subtensor).  The contracted set is walked as
// a sequence of "K boxes": the first kj indices of I_k in full, a block of
// tj values of index kj, and one point of every later index -- a sub-tensor
// of fixed shape slid along the contracted indices (Sec. 3.2.1, Eq. 5-6).
#pragma once
#include <stdint.h>

namespace gett {

constexpr int kMaxDims = 16;   // per index set (== GETT_MAX_RANK)

// Gather modes of an operand tile (see kernel.hpp).
enum GatherMode : int {
    kGatherRowVec = 0,   // 16-byte vectors along the tile's free index (stride-one there)
    kGatherKVec = 1,     // 16-byte vectors along the contracted index (stride-one there)
    kGatherScalar = 2,   // one element per access
    // Column operand only: 16-byte vectors along the operand's stride-one
    // index when that index is the second of the tile's free indices (after
    // a block of C's stride-one index) or the second of the K box (after a
    // block of the row operand's stride-one index); consecutive elements of a
    // vector are KDesc::yes tile rows or K positions apart.
    kGatherRowVecStrided = 3,
    kGatherKVecStrided = 4
};

struct KDesc {
    // ---- free sets, linearised ----
    int64_t sizeX;                 // S_{I_x}
    int64_t sizeY;                 // S_{I_y}
    int32_t nx, ny;                // number of (merged) indices in each set
    int32_t extX[kMaxDims];        // extents, first = fastest in the linear order
    int32_t extY[kMaxDims];
    int64_t strXop[kMaxDims];      // stride of each x index in X
    int64_t strCx[kMaxDims];       // stride of each x index in C
    int64_t strYop[kMaxDims];      // stride of each y index in Y
    int64_t strCy[kMaxDims];       // stride of each y index in C
    // ---- contracted set, walked as K boxes ----
    int32_t nk;                    // number of (merged) contracted indices (>= 1)
    int32_t extK[kMaxDims];
    int64_t strXk[kMaxDims];       // stride of each contracted index in X
    int64_t strYk[kMaxDims];       // stride in Y
    int32_t kj;                    // index that is blocked (earlier ones are whole)
    int32_t tj;                    // block length along index kj
    int32_t kbox;                  // elements in one box = prod(extK[0..kj-1]) * tj
    int32_t nblk;                  // blocks along index kj = ceil(extK[kj] / tj)
    int64_t nsteps;                // boxes = nblk * prod(extK[kj+1..nk-1]); 0 = empty sum
    // ---- grid ----
    int32_t tilesX, tilesY;        // tiles along x and y
    int32_t group;                 // tiles along x that share a column band (L2 reuse)
    int32_t order;                 // 0: banded tile walk, 1: y-fastest walk (C stream order)
    int32_t xcdremap;              // 1: consecutive tiles on one XCD, 0: hardware order
                                   // (-1 in a plan: chosen per call)
    int32_t cvec;                  // 1: C accesses may use 16-byte vectors along y
    int32_t xscalar_kfast;         // scalar gather of X: 1 = contracted index fastest
    int32_t yscalar_kfast;         // scalar gather of Y: 1 = contracted index fastest
    int32_t yes;                   // strided vector gathers of Y: distance between the
                                   // elements of one vector (extent of the first index)
    int32_t kslices;               // workgroups per tile, each summing an equal share of
                                   // the K boxes (1: one per tile); their partial tiles
                                   // are summed in slice order through the workspace
    int32_t crun;                  // > 0: C's stride-one run along y, stored in C order
                                   // through LDS (E elements; 0: per-lane stores only)
    int32_t xperm, yperm;          // > 0: element-wise gathers of X (Y) walk the tile rows
                                   // grouped by row mod this extent (0: in order)
    int32_t tile0;                 // first tile of the grid (> 0: a pass over tiles tile0..)
    // ---- stream-K tail (the tail kernel only) ----
    int32_t tailFull;              // tiles computed whole, one workgroup each
    int32_t tailWgs;               // workgroups that share the boxes of the other tiles
    int32_t tailLen;               // boxes per such workgroup
};

}  // namespace gett
