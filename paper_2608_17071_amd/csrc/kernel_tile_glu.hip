// Tile-kernel launcher of the bf16 SwiGLU projection.
#include "tile_kernel.h"

namespace kernelarc {

hipError_t launch_tile_glu(int cfg, const GluProblem &p, int split, int64_t full_tiles, const Workspace *ws,
                           hipStream_t s) {
    return with_cfg(cfg, [&](auto c, int) {
        using C = decltype(c);
        if constexpr (std::is_same<C, std::nullptr_t>::value) return hipErrorInvalidValue;
        else return launch_cfg_glu<C>(p, 8, split, full_tiles, ws, s);
    });
}

}  // namespace kernelarc
