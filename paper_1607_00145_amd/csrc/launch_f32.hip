// launch_f32.hip -- f32 instantiations of the macro-kernel.
//
// Built once per tile shape with GETT_TILE defined (that tile's launchers:
// every gather-mode pair and kernel kind), and once without it (the table
// that dispatches on the tile).
#include "launch.hpp"

namespace gett {

#ifdef GETT_TILE
template <> LaunchFn pick_tile<float, GETT_TILE>(int xm, int ym, int kind)
{
    return pick_modes<float, GETT_TILE>(xm, ym, kind);
}
#else
template <> LaunchFn pick_tile<float, 0>(int, int, int);
template <> LaunchFn pick_tile<float, 1>(int, int, int);
template <> LaunchFn pick_tile<float, 2>(int, int, int);
template <> LaunchFn pick_tile<float, 3>(int, int, int);
template <> LaunchFn pick_tile<float, 4>(int, int, int);
template <> LaunchFn pick_tile<float, 5>(int, int, int);
template <> LaunchFn pick_tile<float, 6>(int, int, int);
template <> LaunchFn pick_tile<float, 7>(int, int, int);
template <> LaunchFn pick_tile<float, 8>(int, int, int);

LaunchFn launch_fn_f32(int tile, int xm, int ym, int kind)
{
    static_assert(kNumTilesF32 == 9, "update the tile switch");
    switch (tile) {
    case 0: return pick_tile<float, 0>(xm, ym, kind);
    case 1: return pick_tile<float, 1>(xm, ym, kind);
    case 2: return pick_tile<float, 2>(xm, ym, kind);
    case 3: return pick_tile<float, 3>(xm, ym, kind);
    case 4: return pick_tile<float, 4>(xm, ym, kind);
    case 5: return pick_tile<float, 5>(xm, ym, kind);
    case 6: return pick_tile<float, 6>(xm, ym, kind);
    case 7: return pick_tile<float, 7>(xm, ym, kind);
    case 8: return pick_tile<float, 8>(xm, ym, kind);
    }
    return nullptr;
}
#endif

}  // namespace gett
