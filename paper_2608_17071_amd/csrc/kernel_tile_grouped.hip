// Tile-kernel launchers of the grouped (per-expert) forms.
#include "tile_kernel.h"

namespace kernelarc {

hipError_t launch_tile_grouped(int cfg, const Grouped<DenseProblem> &p, hipStream_t s) {
    return with_cfg(cfg, [&](auto c, int) {
        using C = decltype(c);
        if constexpr (std::is_same<C, std::nullptr_t>::value) return hipErrorInvalidValue;
        else return launch_cfg_grouped<C>(p, s);
    });
}

hipError_t launch_tile_grouped_glu(int cfg, const Grouped<GluProblem> &p, hipStream_t s) {
    return with_cfg(cfg, [&](auto c, int) {
        using C = decltype(c);
        if constexpr (std::is_same<C, std::nullptr_t>::value) return hipErrorInvalidValue;
        else return launch_cfg_grouped<C>(p, s);
    });
}

}  // namespace kernelarc
