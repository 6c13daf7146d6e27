// launch_f64.hip -- fp64 instantiations of the macro-kernel.
#include "launch.hpp"

namespace gett {

LaunchFn launch_fn_f64(int tile, int xm, int ym)
{
    static_assert(kNumTilesF64 == 6, "update the tile switch");
    switch (tile) {
    case 0: return pick_modes<double, 0>(xm, ym);
    case 1: return pick_modes<double, 1>(xm, ym);
    case 2: return pick_modes<double, 2>(xm, ym);
    case 3: return pick_modes<double, 3>(xm, ym);
    case 4: return pick_modes<double, 4>(xm, ym);
    case 5: return pick_modes<double, 5>(xm, ym);
    }
    return nullptr;
}

}  // namespace gett
