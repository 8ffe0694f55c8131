// Route kernel instances for f32 inputs, 2-wave tiles.
#include "rr_route_impl.hpp"

namespace rr {

hipError_t launch_route_f32_w2(const RouteArgs &a, int grid, hipStream_t stream)
{
    return route_detail::launch_family<float, 2>(a, grid, stream);
}

}  // namespace rr
