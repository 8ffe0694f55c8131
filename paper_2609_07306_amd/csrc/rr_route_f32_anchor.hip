// Route kernel instances: f32 inputs, anchor routing.
#include "rr_route_impl.hpp"

namespace rr {

hipError_t launch_route_f32_anchor(const RouteArgs &a, int grid, hipStream_t stream)
{
    return route_detail::launch_family<MODE_ANCHOR, float>(a, grid, stream);
}

}  // namespace rr
