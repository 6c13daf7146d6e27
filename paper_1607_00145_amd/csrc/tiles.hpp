// tiles.hpp -- the macro-kernel tile shapes compiled into the library.
//
// A tile is MT x NT elements of C (x by y) computed by one workgroup of
// WM x WN wavefronts (64 lanes each); each K box holds up to KT contracted
// elements.  These play the role of the paper's blocking parameters
// m_C, n_C, k_C (Sec. 3.3); the register tile of one wavefront,
// (MT/WM) x (NT/WN) built from 16x16 MFMA blocks, plays the role of
// m_R x n_R (Sec. 3.1).  RX / RY are the rows each lane reads from LDS at
// once on the x / y side (1, or 16 bytes' worth).  `eff` is the fraction of
// the MFMA peak the tile sustains when compute-bound, used by the analyser's
// cost model (measured on MI355X).
#pragma once

namespace gett {

struct TileShape {
    int mt, nt, kt, wm, wn, rx, ry;
    float eff;
};

constexpr TileShape kTilesF32[] = {
    {128, 128, 16, 2, 2, 4, 4, 0.80f},
    {64, 64, 16, 1, 1, 4, 4, 0.40f},
};
constexpr TileShape kTilesF64[] = {
    {128, 128, 16, 2, 2, 2, 2, 0.60f},
    {64, 64, 16, 1, 1, 2, 2, 0.30f},
    {144, 144, 16, 3, 3, 1, 1, 0.70f},
    {128, 64, 8, 2, 2, 2, 2, 0.50f},
};
constexpr int kNumTilesF32 = sizeof(kTilesF32) / sizeof(kTilesF32[0]);
constexpr int kNumTilesF64 = sizeof(kTilesF64) / sizeof(kTilesF64[0]);
constexpr int kNumGatherModes = 3;

}  // namespace gett
