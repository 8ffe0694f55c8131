// Route kernel instances: f32 inputs, full routing.
#include "rr_route_impl.hpp"

namespace rr {

hipError_t launch_route_f32_full(const RouteArgs &a, int grid, hipStream_t stream)
{
    return route_detail::launch_family<MODE_FULL, float>(a, grid, stream);
}

}  // namespace rr
