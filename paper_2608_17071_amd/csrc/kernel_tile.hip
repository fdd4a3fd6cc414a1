// Tile-kernel launchers of the bf16 linear layer (plain and general forms)
// and the host-side configuration queries.
#include "tile_kernel.h"

namespace kernelarc {

TileShape tile_shape(int cfg) {
    return with_cfg(cfg, [](auto c, int per_cu) {
        using C = decltype(c);
        if constexpr (std::is_same<C, std::nullptr_t>::value) return TileShape{0, 0, 0, 0};
        else return TileShape{C::BM, C::BN, C::BK, per_cu};
    });
}

bool tile_glu_ok(int cfg) {
    return with_cfg(cfg, [](auto c, int) {
        using C = decltype(c);
        if constexpr (std::is_same<C, std::nullptr_t>::value) return false;
        else return glu_ok<C>();
    });
}

bool tile_is_m16(int cfg) {
    return with_cfg(cfg, [](auto c, int) {
        using C = decltype(c);
        if constexpr (std::is_same<C, std::nullptr_t>::value) return false;
        else return C::M16;
    });
}

bool tile_f8_ok(int cfg) {
    return with_cfg(cfg, [](auto c, int) {
        using C = decltype(c);
        if constexpr (std::is_same<C, std::nullptr_t>::value) return false;
        else return f8_ok<C>();
    });
}

hipError_t launch_tile(int cfg, const Problem &p, int split, int64_t full_tiles, const Workspace *ws,
                       hipStream_t s) {
    return with_cfg(cfg, [&](auto c, int) {
        using C = decltype(c);
        if constexpr (std::is_same<C, std::nullptr_t>::value) return hipErrorInvalidValue;
        else return launch_cfg<C>(p, 8, split, full_tiles, ws, s);
    });
}

}  // namespace kernelarc
