// launch_f32.hip -- fp32 instantiations of the macro-kernel.
#include "launch.hpp"

namespace gett {

LaunchFn launch_fn_f32(int tile, int xm, int ym, int kind)
{
    static_assert(kNumTilesF32 == 7, "update the tile switch");
    switch (tile) {
    case 0: return pick_modes<float, 0>(xm, ym, kind);
    case 1: return pick_modes<float, 1>(xm, ym, kind);
    case 2: return pick_modes<float, 2>(xm, ym, kind);
    case 3: return pick_modes<float, 3>(xm, ym, kind);
    case 4: return pick_modes<float, 4>(xm, ym, kind);
    case 5: return pick_modes<float, 5>(xm, ym, kind);
    case 6: return pick_modes<float, 6>(xm, ym, kind);
    }
    return nullptr;
}

}  // namespace gett
