// launch.hpp -- host launchers for every compiled (dtype, tile, gather mode)
// combination.  Included by one .hip file per dtype.
#pragma once
#include <hip/hip_runtime.h>

#include <atomic>

#include "direct.hpp"
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

// Workgroups of a persistent kernel: as many as fit on the device at once,
// and no more than there are tiles.  The count per device is looked up once
// per kernel (the first launch on each device, up to 64 devices); the cache
// lives in the instantiation for that kernel, since kernels that share a
// signature can differ in occupancy.
template <auto kernel>
unsigned persistent_grid(int threads, unsigned tiles, size_t lds = 0)
{
    static std::atomic<int> cached[64];   // CUs x workgroups per CU, 0: not yet known
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess) return 0;
    int n = dev >= 0 && dev < 64 ? cached[dev].load(std::memory_order_relaxed) : 0;
    if (n <= 0) {
        int cus = 0, per = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
            return 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per, kernel, threads, lds) != hipSuccess)
            return 0;
        n = cus * (per > 0 ? per : 1);
        if (dev >= 0 && dev < 64) cached[dev].store(n, std::memory_order_relaxed);
    }
    return (unsigned)n < tiles ? (unsigned)n : tiles;
}

// Let the kernel take `bytes` of dynamic LDS (above the default cap), once per
// kernel and device (up to 64 devices; a later device asks again).  The flag
// lives in the instantiation for that kernel: kernels that share a signature
// each ask for themselves.
template <auto kernel>
hipError_t allow_dynamic_lds(size_t bytes)
{
    static std::atomic<int> done[64];
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev >= 0 && dev < 64 && done[dev].load(std::memory_order_relaxed)) return hipSuccess;
    e = hipFuncSetAttribute(reinterpret_cast<const void *>(kernel),
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
    if (e == hipSuccess && dev >= 0 && dev < 64) done[dev].store(1, std::memory_order_relaxed);
    return e;
}

template <typename T, int TI, int XM, int YM, int KIND>
hipError_t launch_one(const KDesc &d, const void *X, const void *Y, void *C, double alpha,
                      double beta, const Partials &w, hipStream_t stream)
{
    if ((KIND == 2 || KIND == 3) && (!w.tiles || !w.counters))
        return hipErrorInvalidValue;   // partial tiles need the workspace
    constexpr TileShape t = TileTable<T>::tiles[TI];
    const unsigned tiles = (unsigned)d.tilesX * (unsigned)d.tilesY;
    if (tiles == 0) return hipSuccess;
    const int threads = t.wm * t.wn * 64;
    if constexpr (KIND == 0) {
        if (d.kslices > 1) return hipErrorInvalidValue;   // the sliced variant (kind 2) does those
        if ((unsigned)d.tile0 >= tiles) return hipSuccess;
        hipLaunchKernelGGL(
            (gett_macro_kernel<T, t.mt, t.nt, t.kt, t.wm, t.wn, t.rx, t.ry, t.wpe, t.pf, t.nbuf, XM,
                               YM, t.onebox, t.corder>),
            dim3(tiles - (unsigned)d.tile0), dim3(threads), 0, stream, d,
            static_cast<const T *>(X), static_cast<const T *>(Y), static_cast<T *>(C),
            static_cast<T>(alpha), static_cast<T>(beta), static_cast<T *>(nullptr), nullptr);
    } else if constexpr (KIND == 2) {
        if (d.kslices < 2 || d.tile0 != 0) return hipErrorInvalidValue;
        hipLaunchKernelGGL(
            (gett_macro_kernel<T, t.mt, t.nt, t.kt, t.wm, t.wn, t.rx, t.ry, t.wpe, t.pf, t.nbuf, XM,
                               YM, t.onebox, t.corder, 0, 1>),
            dim3(tiles * (unsigned)d.kslices), dim3(threads), 0, stream, d,
            static_cast<const T *>(X), static_cast<const T *>(Y), static_cast<T *>(C),
            static_cast<T>(alpha), static_cast<T>(beta), static_cast<T *>(w.tiles), w.counters);
    } else if constexpr (KIND == 3) {
        if (d.tailFull < 0 || d.tailWgs < 1 || d.tailLen < 1 || (unsigned)d.tailFull >= tiles ||
            (uint64_t)d.tailWgs * (uint64_t)d.tailLen <
                (uint64_t)(tiles - (unsigned)d.tailFull) * (uint64_t)d.nsteps)
            return hipErrorInvalidValue;   // the tail workgroups must cover every box
        hipLaunchKernelGGL(
            (gett_macro_kernel<T, t.mt, t.nt, t.kt, t.wm, t.wn, t.rx, t.ry, t.wpe, t.pf, t.nbuf, XM,
                               YM, t.onebox, t.corder, 1>),
            dim3((unsigned)d.tailFull + (unsigned)d.tailWgs), dim3(threads), 0, stream, d,
            static_cast<const T *>(X), static_cast<const T *>(Y), static_cast<T *>(C),
            static_cast<T>(alpha), static_cast<T>(beta), static_cast<T *>(w.tiles), w.counters);
    } else if constexpr (KIND == 4) {
        if (d.kslices > 1) return hipErrorInvalidValue;   // whole tiles only
        if ((unsigned)d.tile0 >= tiles) return hipSuccess;
        // every piece of every box inside the tensors: the variant without checks
        const bool whole = d.sizeX % t.mt == 0 && d.sizeY % t.nt == 0 &&
                           (d.nsteps == 0 || (d.kbox == t.kt && d.extK[d.kj] % d.tj == 0));
        constexpr auto kWhole =
            gett_direct_kernel<T, t.mt, t.nt, t.kt, t.wm, t.wn, t.rx, t.ry, XM, YM, true>;
        constexpr auto kPart =
            gett_direct_kernel<T, t.mt, t.nt, t.kt, t.wm, t.wn, t.rx, t.ry, XM, YM, false>;
        constexpr size_t lds = 2 * (size_t)(t.mt + t.nt) * t.kt * sizeof(T);
        const auto k = whole ? kWhole : kPart;
        const hipError_t e =
            whole ? allow_dynamic_lds<kWhole>(lds) : allow_dynamic_lds<kPart>(lds);
        if (e != hipSuccess) return e;
        hipLaunchKernelGGL(
            k, dim3(tiles - (unsigned)d.tile0), dim3(threads), lds, stream, d,
            static_cast<const T *>(X), static_cast<const T *>(Y), static_cast<T *>(C),
            static_cast<T>(alpha), static_cast<T>(beta));
    } else if constexpr (KIND == 5) {
        if (d.kslices > 1 || d.nsteps != 1) return hipErrorInvalidValue;   // one K box
        if ((unsigned)d.tile0 >= tiles) return hipSuccess;
        const bool whole = d.sizeX % t.mt == 0 && d.sizeY % t.nt == 0 && d.kbox == t.kt &&
                           d.extK[d.kj] % d.tj == 0;
        constexpr auto kWhole =
            gett_direct_stream_kernel<T, t.mt, t.nt, t.kt, t.wm, t.wn, t.rx, t.ry, XM, YM, true>;
        constexpr auto kPart =
            gett_direct_stream_kernel<T, t.mt, t.nt, t.kt, t.wm, t.wn, t.rx, t.ry, XM, YM, false>;
        constexpr size_t lds = 2 * (size_t)(t.mt + t.nt) * t.kt * sizeof(T);
        const auto k = whole ? kWhole : kPart;
        hipError_t e = whole ? allow_dynamic_lds<kWhole>(lds) : allow_dynamic_lds<kPart>(lds);
        if (e != hipSuccess) return e;
        const unsigned left = tiles - (unsigned)d.tile0;
        const unsigned grid = whole ? persistent_grid<kWhole>(threads, left, lds)
                                    : persistent_grid<kPart>(threads, left, lds);
        if (grid == 0) return hipErrorInvalidValue;
        hipLaunchKernelGGL(k, dim3(grid), dim3(threads), lds, stream, d,
                           static_cast<const T *>(X), static_cast<const T *>(Y),
                           static_cast<T *>(C), static_cast<T>(alpha), static_cast<T>(beta));
    } else {
        constexpr auto k =
            gett_stream_kernel<T, t.mt, t.nt, t.kt, t.wm, t.wn, t.rx, t.ry, t.stream, XM, YM>;
        const unsigned grid = persistent_grid<k>(threads, tiles);
        if (grid == 0) return hipErrorInvalidValue;
        hipLaunchKernelGGL(k, dim3(grid), dim3(threads), 0, stream, d,
                           static_cast<const T *>(X), static_cast<const T *>(Y),
                           static_cast<T *>(C), static_cast<T>(alpha), static_cast<T>(beta));
    }
    return hipGetLastError();
}

template <typename T, int TI>
LaunchFn pick_modes(int xm, int ym, int kind)
{
    constexpr bool kStream = TileTable<T>::tiles[TI].stream != 0;
    constexpr bool kTail = TileTable<T>::tiles[TI].tail != 0;
    constexpr bool kDirect = TileTable<T>::tiles[TI].deff > 0.0f;
    constexpr bool kDStream = TileTable<T>::tiles[TI].dsbw > 0.0f;
#define GETT_CASE(a, b)                                                                       \
    if (xm == a && ym == b) {                                                                 \
        constexpr bool kDir = kDirect && a <= 1 && b <= 1;   /* vector gathers only */       \
        if (kind == 0) return &launch_one<T, TI, a, b, 0>;                                   \
        if (kind == 2) return &launch_one<T, TI, a, b, 2>;                                   \
        if (kind == 1 && kStream) return &launch_one<T, TI, a, b, kStream ? 1 : 0>;          \
        if (kind == 3 && kTail) return &launch_one<T, TI, a, b, kTail ? 3 : 0>;              \
        if (kind == 4 && kDir) return &launch_one<T, TI, a, b, kDir ? 4 : 0>;                \
        constexpr bool kDS = kDStream && a <= 1 && b <= 1;                                    \
        if (kind == 5 && kDS) return &launch_one<T, TI, a, b, kDS ? 5 : 0>;                  \
        return nullptr;                                                                       \
    }
    GETT_CASE(0, 0) GETT_CASE(0, 1) GETT_CASE(0, 2) GETT_CASE(0, 3) GETT_CASE(0, 4)
    GETT_CASE(1, 0) GETT_CASE(1, 1) GETT_CASE(1, 2) GETT_CASE(1, 3) GETT_CASE(1, 4)
    GETT_CASE(2, 0) GETT_CASE(2, 1) GETT_CASE(2, 2) GETT_CASE(2, 3) GETT_CASE(2, 4)
#undef GETT_CASE
    return nullptr;
}

// The launchers of one tile shape.  Each (dtype, tile) pair is compiled in a
// translation unit of its own (launch_f32.hip / launch_f64.hip built once per
// tile with GETT_TILE defined), so the instantiations build in parallel.
template <typename T, int TI> LaunchFn pick_tile(int xm, int ym, int kind);

}  // namespace gett
