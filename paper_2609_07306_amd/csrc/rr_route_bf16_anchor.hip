// Route kernel instances: bf16 inputs, anchor routing.
#include "rr_route_impl.hpp"

namespace rr {

hipError_t launch_route_bf16_anchor(const RouteArgs &a, int grid, hipStream_t stream)
{
    return route_detail::launch_family<MODE_ANCHOR, bf16_t>(a, grid, stream);
}

}  // namespace rr
