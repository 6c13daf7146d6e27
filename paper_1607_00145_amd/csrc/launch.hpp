// launch.hpp -- host launchers for every compiled (dtype, tile, gather mode)
// combination.  Included by one .hip file per dtype.
#pragma once
#include <hip/hip_runtime.h>

#include "kernel.hpp"
#include "plan.hpp"
#include "tiles.hpp"

namespace gett {

template <typename T> struct TileTable;
template <> struct TileTable<float> {
    static constexpr const TileShape *tiles = kTilesF32;
    static constexpr int n = kNumTilesF32;
};
template <> struct TileTable<double> {
    static constexpr const TileShape *tiles = kTilesF64;
    static constexpr int n = kNumTilesF64;
};

template <typename T, int TI, int XM, int YM>
hipError_t launch_one(const KDesc &d, const void *X, const void *Y, void *C, double alpha,
                      double beta, hipStream_t stream)
{
    constexpr TileShape t = TileTable<T>::tiles[TI];
    const unsigned grid = (unsigned)d.tilesX * (unsigned)d.tilesY;
    if (grid == 0) return hipSuccess;
    hipLaunchKernelGGL((gett_macro_kernel<T, t.mt, t.nt, t.kt, t.wm, t.wn, t.rx, t.ry, t.wpe, XM, YM>),
                       dim3(grid),
                       dim3(t.wm * t.wn * 64), 0, stream, d, static_cast<const T *>(X),
                       static_cast<const T *>(Y), static_cast<T *>(C), static_cast<T>(alpha),
                       static_cast<T>(beta));
    return hipGetLastError();
}

template <typename T, int TI>
LaunchFn pick_modes(int xm, int ym)
{
#define GETT_CASE(a, b) \
    if (xm == a && ym == b) return &launch_one<T, TI, a, b>;
    GETT_CASE(0, 0) GETT_CASE(0, 1) GETT_CASE(0, 2)
    GETT_CASE(1, 0) GETT_CASE(1, 1) GETT_CASE(1, 2)
    GETT_CASE(2, 0) GETT_CASE(2, 1) GETT_CASE(2, 2)
#undef GETT_CASE
    return nullptr;
}

}  // namespace gett
