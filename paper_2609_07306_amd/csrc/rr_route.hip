// Dispatch of the GEMM + TopK route kernel (rr_route_impl.hpp) by input type
// and tile width.
#include "rr_internal.hpp"

namespace rr {

hipError_t launch_route_f32_w2(const RouteArgs &a, int grid, hipStream_t stream);
hipError_t launch_route_f32_w4(const RouteArgs &a, int grid, hipStream_t stream);
hipError_t launch_route_bf16_w2(const RouteArgs &a, int grid, hipStream_t stream);
hipError_t launch_route_bf16_w4(const RouteArgs &a, int grid, hipStream_t stream);

bool route_supported(int dtype, int d, int T)
{
    if (T < 1 || T > 128) return false;
    if (dtype == 0) return d == 32 || d == 64 || d == 128;
    if (dtype == 1) return d == 32 || d == 64 || d == 128 || d == 256;
    return false;
}

int route_tile_rows(int mode) { return mode == MODE_REROUTE ? 32 * kRerouteWaves : 32 * kFullWaves; }

hipError_t launch_route(const RouteArgs &a, int dtype, int grid, hipStream_t stream)
{
    static_assert(kRerouteWaves == 2 && kFullWaves == 4, "instantiated tile widths");
    const bool reroute = a.mode == MODE_REROUTE;
    if (dtype == 0) return reroute ? launch_route_f32_w2(a, grid, stream) : launch_route_f32_w4(a, grid, stream);
    return reroute ? launch_route_bf16_w2(a, grid, stream) : launch_route_bf16_w4(a, grid, stream);
}

}  // namespace rr
