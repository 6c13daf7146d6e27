// launch_f64.hip -- fp64 instantiations of the macro-kernel.
#include "launch.hpp"

namespace gett {

LaunchFn launch_fn_f64(int tile, int xm, int ym, int kind)
{
    static_assert(kNumTilesF64 == 15, "update the tile switch");
    switch (tile) {
    case 0: return pick_modes<double, 0>(xm, ym, kind);
    case 1: return pick_modes<double, 1>(xm, ym, kind);
    case 2: return pick_modes<double, 2>(xm, ym, kind);
    case 3: return pick_modes<double, 3>(xm, ym, kind);
    case 4: return pick_modes<double, 4>(xm, ym, kind);
    case 5: return pick_modes<double, 5>(xm, ym, kind);
    case 6: return pick_modes<double, 6>(xm, ym, kind);
    case 7: return pick_modes<double, 7>(xm, ym, kind);
    case 8: return pick_modes<double, 8>(xm, ym, kind);
    case 9: return pick_modes<double, 9>(xm, ym, kind);
    case 10: return pick_modes<double, 10>(xm, ym, kind);
    case 11: return pick_modes<double, 11>(xm, ym, kind);
    case 12: return pick_modes<double, 12>(xm, ym, kind);
    case 13: return pick_modes<double, 13>(xm, ym, kind);
    case 14: return pick_modes<double, 14>(xm, ym, kind);
    }
    return nullptr;
}

}  // namespace gett
