// launch_f64.hip -- f64 instantiations of the macro-kernel.
//
// Built once per tile shape with GETT_TILE defined (that tile's launchers:
// every gather-mode pair and kernel kind), and once without it (the table
// that dispatches on the tile).
#include "launch.hpp"

namespace gett {

#ifdef GETT_TILE
template <> LaunchFn pick_tile<double, GETT_TILE>(int xm, int ym, int kind)
{
    return pick_modes<double, GETT_TILE>(xm, ym, kind);
}
#else
template <> LaunchFn pick_tile<double, 0>(int, int, int);
template <> LaunchFn pick_tile<double, 1>(int, int, int);
template <> LaunchFn pick_tile<double, 2>(int, int, int);
template <> LaunchFn pick_tile<double, 3>(int, int, int);
template <> LaunchFn pick_tile<double, 4>(int, int, int);
template <> LaunchFn pick_tile<double, 5>(int, int, int);
template <> LaunchFn pick_tile<double, 6>(int, int, int);
template <> LaunchFn pick_tile<double, 7>(int, int, int);
template <> LaunchFn pick_tile<double, 8>(int, int, int);
template <> LaunchFn pick_tile<double, 9>(int, int, int);
template <> LaunchFn pick_tile<double, 10>(int, int, int);
template <> LaunchFn pick_tile<double, 11>(int, int, int);
template <> LaunchFn pick_tile<double, 12>(int, int, int);
template <> LaunchFn pick_tile<double, 13>(int, int, int);
template <> LaunchFn pick_tile<double, 14>(int, int, int);

LaunchFn launch_fn_f64(int tile, int xm, int ym, int kind)
{
    static_assert(kNumTilesF64 == 15, "update the tile switch");
    switch (tile) {
    case 0: return pick_tile<double, 0>(xm, ym, kind);
    case 1: return pick_tile<double, 1>(xm, ym, kind);
    case 2: return pick_tile<double, 2>(xm, ym, kind);
    case 3: return pick_tile<double, 3>(xm, ym, kind);
    case 4: return pick_tile<double, 4>(xm, ym, kind);
    case 5: return pick_tile<double, 5>(xm, ym, kind);
    case 6: return pick_tile<double, 6>(xm, ym, kind);
    case 7: return pick_tile<double, 7>(xm, ym, kind);
    case 8: return pick_tile<double, 8>(xm, ym, kind);
    case 9: return pick_tile<double, 9>(xm, ym, kind);
    case 10: return pick_tile<double, 10>(xm, ym, kind);
    case 11: return pick_tile<double, 11>(xm, ym, kind);
    case 12: return pick_tile<double, 12>(xm, ym, kind);
    case 13: return pick_tile<double, 13>(xm, ym, kind);
    case 14: return pick_tile<double, 14>(xm, ym, kind);
    }
    return nullptr;
}
#endif

}  // namespace gett
