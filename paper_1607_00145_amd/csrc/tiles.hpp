// tiles.hpp -- the macro-kernel tile shapes compiled into the library.
//
// A tile is MT x NT elements of C (x by y) computed by one workgroup of
// WM x WN wavefronts (64 lanes each); each K box holds up to KT contracted
// elements.  These play the role of the paper's blocking parameters
// m_C, n_C, k_C (Sec. 3.3); the register tile of one wavefront,
// (MT/WM) x (NT/WN) built from 16x16 MFMA blocks, plays the role of
// m_R x n_R (Sec. 3.1).  RX / RY are the rows each lane reads from LDS at
// once on the x / y side (1, or 16 bytes' worth).  `eff` and `bw` feed the
// analyser's cost model; they were measured on MI355X with the workloads of
// the benchmark.
#pragma once

namespace gett {

struct TileShape {
    int mt, nt, kt, wm, wn, rx, ry;
    int wpe;     // minimum wavefronts per SIMD the register allocation must allow
    int pf;      // K boxes gathered ahead of the MFMAs (1 or 2 register stages)
    int nbuf;    // LDS buffers for the packed tiles (1 or 2)
    int stream;  // > 0: also compiled as the persistent streaming kernel, with this
                 // minimum number of wavefronts per SIMD
    float eff;   // fraction of the MFMA peak sustained when compute-bound
    float bw;    // fraction of the HBM peak sustained when streaming C (macro-kernel)
    float sbw;   // the same for the streaming kernel
    int onebox;  // 1: no prefetch (each box gathered, packed and multiplied in turn),
                 // for contracted sets that fit one K box; fewer registers live at once
    int corder;  // 1: the kernel carries the C-order epilogue (unpack_c_order)
    int tail;    // 1: also compiled as the stream-K tail kernel
    float deff;  // > 0: also compiled as the direct-load kernel (operands copied
                 // straight into LDS), which sustains this fraction of the MFMA
                 // peak when compute-bound
    float dsbw;  // > 0: also compiled as the persistent direct-load kernel for
                 // plans whose contracted set is one K box, which sustains this
                 // fraction of the HBM peak when streaming C
};

constexpr TileShape kTilesF32[] = {
    {128, 128, 16, 2, 2, 4, 4, 1, 1, 2, 0, 0.75f, 0.61f, 0.0f, 0, 1},
    {64, 64, 16, 1, 1, 4, 4, 1, 1, 2, 0, 0.67f, 0.62f, 0.0f, 0, 1},
    {128, 128, 16, 2, 2, 4, 4, 3, 1, 2, 2, 0.71f, 0.675f, 0.64f, 0, 1, 1},
    {64, 256, 16, 1, 4, 4, 4, 3, 1, 2, 2, 0.70f, 0.70f, 0.63f, 0, 1},
    {128, 128, 32, 2, 2, 4, 4, 1, 1, 2, 0, 0.806f, 0.61f, 0.0f, 0, 1, 0, 0.87f},
    {64, 32, 32, 2, 2, 2, 1, 2, 2, 2, 0, 0.64f, 0.35f, 0.0f},
    {32, 64, 32, 2, 2, 1, 2, 2, 2, 2, 0, 0.65f, 0.35f, 0.0f},
    {256, 128, 32, 4, 2, 4, 4, 2, 1, 2, 0, 0.75f, 0.55f, 0.0f, 0, 0, 0, 0.89f},
    {128, 256, 32, 2, 4, 4, 4, 2, 1, 2, 0, 0.75f, 0.55f, 0.0f, 0, 0, 0, 0.89f},
};
constexpr TileShape kTilesF64[] = {
    {128, 128, 16, 2, 2, 2, 2, 1, 2, 2, 0, 0.65f, 0.34f, 0.0f},
    {64, 64, 16, 1, 1, 2, 2, 1, 2, 2, 0, 0.59f, 0.32f, 0.0f},
    {144, 144, 16, 3, 3, 1, 1, 1, 2, 2, 0, 0.79f, 0.36f, 0.0f},
    {128, 64, 8, 2, 2, 2, 2, 3, 1, 2, 2, 0.70f, 0.53f, 0.53f},
    {128, 64, 24, 2, 2, 2, 2, 2, 1, 2, 2, 0.69f, 0.49f, 0.51f},
    {64, 64, 16, 2, 2, 2, 2, 2, 2, 2, 0, 0.75f, 0.34f, 0.0f},
    {64, 128, 16, 2, 2, 2, 2, 2, 2, 2, 0, 0.785f, 0.34f, 0.0f},
    {128, 64, 16, 2, 2, 2, 2, 2, 2, 2, 0, 0.785f, 0.34f, 0.0f},
    {96, 128, 16, 2, 2, 1, 2, 2, 2, 2, 0, 0.79f, 0.34f, 0.0f, 0, 0, 1},
    {128, 64, 24, 2, 2, 2, 2, 3, 1, 1, 0, 0.785f, 0.615f, 0.0f, 0, 0, 1},
    {64, 128, 24, 1, 4, 2, 2, 3, 1, 1, 0, 0.775f, 0.59f, 0.0f},
    {64, 128, 24, 2, 2, 2, 2, 3, 1, 1, 0, 0.785f, 0.668f, 0.0f, 0, 0, 1},
    {64, 32, 16, 2, 2, 2, 1, 2, 2, 2, 0, 0.70f, 0.485f, 0.0f},
    {32, 64, 16, 2, 2, 1, 2, 2, 2, 2, 0, 0.71f, 0.49f, 0.0f},
    {64, 128, 24, 2, 2, 2, 2, 4, 1, 1, 0, 0.785f, 0.70f, 0.0f, 1, 0, 0, 0.0f, 0.75f},
};
constexpr int kNumTilesF32 = sizeof(kTilesF32) / sizeof(kTilesF32[0]);
constexpr int kNumTilesF64 = sizeof(kTilesF64) / sizeof(kTilesF64[0]);
constexpr int kNumGatherModes = 5;

}  // namespace gett
