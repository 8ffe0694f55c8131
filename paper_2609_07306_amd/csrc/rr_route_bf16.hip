// Route kernel instances for bf16 inputs.
#include "rr_route_impl.hpp"

namespace rr {

hipError_t launch_route_bf16(const RouteArgs &a, int grid, hipStream_t stream)
{
    return route_detail::launch_family<bf16_t>(a, grid, stream);
}

}  // namespace rr
