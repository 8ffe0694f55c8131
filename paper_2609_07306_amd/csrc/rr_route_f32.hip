// Route kernel instances for f32 inputs.
#include "rr_route_impl.hpp"

namespace rr {

hipError_t launch_route_f32(const RouteArgs &a, int grid, hipStream_t stream)
{
    return route_detail::launch_family<float>(a, grid, stream);
}

}  // namespace rr
