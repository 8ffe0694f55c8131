// Route kernel instances for bf16 inputs, 4-wave tiles.
#include "rr_route_impl.hpp"

namespace rr {

hipError_t launch_route_bf16_w4(const RouteArgs &a, int grid, hipStream_t stream)
{
    return route_detail::launch_family<bf16_t, 4>(a, grid, stream);
}

}  // namespace rr
