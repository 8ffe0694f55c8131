// Dispatch of the GEMM + TopK route kernel (rr_route_impl.hpp) by mode, input
// type and tile width.
#include "rr_route_impl.hpp"

namespace rr {

hipError_t launch_route_f32_full(const RouteArgs &a, int grid, hipStream_t stream);
hipError_t launch_route_f32_anchor(const RouteArgs &a, int grid, hipStream_t stream);
hipError_t launch_route_f32_reroute(const RouteArgs &a, int grid, hipStream_t stream);
hipError_t launch_route_bf16_full(const RouteArgs &a, int grid, hipStream_t stream);
hipError_t launch_route_bf16_anchor(const RouteArgs &a, int grid, hipStream_t stream);
hipError_t launch_route_bf16_reroute(const RouteArgs &a, int grid, hipStream_t stream);
hipError_t launch_route_f32_relay(const RouteArgs &a, int grid, hipStream_t stream);
hipError_t launch_route_bf16_relay(const RouteArgs &a, int grid, hipStream_t stream);

bool route_supported(int dtype, int d, int T)
{
    if (T < 1 || T > 128) return false;
    if (dtype == 0) return d == 32 || d == 64 || d == 128;
    if (dtype == 1) return d == 32 || d == 64 || d == 128 || d == 256;
    return false;
}

// Fewer 128-row tiles than compute units leave units idle and each tile's
// sweeps long (binary32 products run at 1/16 of the bf16 rate; a causal
// tile's key range is its last row's): 32-row tiles then spread the same
// rows over four times the workgroups.  With a tile per unit or more, the
// extra passes over each key head cost more than they save.
int route_tile_rows(int T, int n_heads, int n_q)
{
    if (T > 64) return kWideTileRows;
    const int64_t narrow = (int64_t)n_heads * ((n_q + kNarrowTileRows - 1) / kNarrowTileRows);
    return narrow < kFewTiles ? kSmallTileRows : kNarrowTileRows;
}

int route_relay_max_bm_words(int dtype, int d, int T)
{
    using route_detail::relay_max_bm_words;
    switch (d) {
    case 32: return dtype == 0 ? relay_max_bm_words<float, 32>(T) : relay_max_bm_words<bf16_t, 32>(T);
    case 64: return dtype == 0 ? relay_max_bm_words<float, 64>(T) : relay_max_bm_words<bf16_t, 64>(T);
    case 128: return dtype == 0 ? relay_max_bm_words<float, 128>(T) : relay_max_bm_words<bf16_t, 128>(T);
    case 256: return dtype == 0 ? 0 : relay_max_bm_words<bf16_t, 256>(T);
    default: return 0;
    }
}

hipError_t launch_route(const RouteArgs &a, int dtype, int grid, hipStream_t stream)
{
    switch (a.mode) {
    case MODE_FULL: return dtype == 0 ? launch_route_f32_full(a, grid, stream) : launch_route_bf16_full(a, grid, stream);
    case MODE_ANCHOR:
        return dtype == 0 ? launch_route_f32_anchor(a, grid, stream) : launch_route_bf16_anchor(a, grid, stream);
    case MODE_REROUTE:
        return dtype == 0 ? launch_route_f32_reroute(a, grid, stream) : launch_route_bf16_reroute(a, grid, stream);
    case MODE_RELAY:
        return dtype == 0 ? launch_route_f32_relay(a, grid, stream) : launch_route_bf16_relay(a, grid, stream);
    default: break;
    }
    return hipErrorInvalidValue;
}

}  // namespace rr
