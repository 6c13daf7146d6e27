// tiles.hpp -- the macro-kernel tile shapes compiled into the library.
//
// A tile is MT x NT elements of C (x by y) computed by one workgroup of
// WM x WN wavefronts (64 lanes each); each step consumes KT contracted
// elements.  These play the role of the paper's blocking parameters
// m_C, n_C, k_C (Sec. 3.3); the register tile of one wavefront plays the
// role of m_R x n_R (Sec. 3.1).
#pragma once

namespace gett {

struct TileShape {
    int mt, nt, kt, wm, wn;
};

// fp32: MFMA 16x16x4 f32 blocks; a wave tile is a multiple of 64 x 64.
constexpr TileShape kTilesF32[] = {
    {128, 128, 16, 2, 2},
    {64, 64, 16, 1, 1},
};
// fp64: MFMA 16x16x4 f64 blocks; a wave tile is a multiple of 32 x 32.
constexpr TileShape kTilesF64[] = {
    {128, 128, 16, 2, 2},
    {64, 64, 16, 1, 1},
};
constexpr int kNumTilesF32 = sizeof(kTilesF32) / sizeof(kTilesF32[0]);
constexpr int kNumTilesF64 = sizeof(kTilesF64) / sizeof(kTilesF64[0]);
constexpr int kNumGatherModes = 3;

}  // namespace gett
