// Route kernel instances: bf16 inputs, reroute routing.
#include "rr_route_impl.hpp"

namespace rr {

hipError_t launch_route_bf16_reroute(const RouteArgs &a, int grid, hipStream_t stream)
{
    return route_detail::launch_family<MODE_REROUTE, bf16_t>(a, grid, stream);
}

}  // namespace rr
