// Dispatch of the GEMM + TopK route kernel (rr_route_impl.hpp) by input type
// and tile width.
#include "rr_internal.hpp"

namespace rr {

hipError_t launch_route_f32_full(const RouteArgs &a, int grid, hipStream_t stream);
hipError_t launch_route_f32_anchor(const RouteArgs &a, int grid, hipStream_t stream);
hipError_t launch_route_f32_reroute(const RouteArgs &a, int grid, hipStream_t stream);
hipError_t launch_route_bf16_full(const RouteArgs &a, int grid, hipStream_t stream);
hipError_t launch_route_bf16_anchor(const RouteArgs &a, int grid, hipStream_t stream);
hipError_t launch_route_bf16_reroute(const RouteArgs &a, int grid, hipStream_t stream);

bool route_supported(int dtype, int d, int T)
{
    if (T < 1 || T > 128) return false;
    if (dtype == 0) return d == 32 || d == 64 || d == 128;
    if (dtype == 1) return d == 32 || d == 64 || d == 128 || d == 256;
    return false;
}

int route_tile_rows(int T) { return T > 64 ? kWideTileRows : kNarrowTileRows; }

hipError_t launch_route(const RouteArgs &a, int dtype, int grid, hipStream_t stream)
{
    switch (a.mode) {
    case MODE_FULL: return dtype == 0 ? launch_route_f32_full(a, grid, stream) : launch_route_bf16_full(a, grid, stream);
    case MODE_ANCHOR:
        return dtype == 0 ? launch_route_f32_anchor(a, grid, stream) : launch_route_bf16_anchor(a, grid, stream);
    case MODE_REROUTE:
        return dtype == 0 ? launch_route_f32_reroute(a, grid, stream) : launch_route_bf16_reroute(a, grid, stream);
    default: break;
    }
    return hipErrorInvalidValue;
}

}  // namespace rr
