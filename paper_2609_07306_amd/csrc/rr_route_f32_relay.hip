// Route kernel instances: f32 inputs, relay layers (rescoring + trigger +
// routing of the flagged rows in one pass).
#include "rr_route_impl.hpp"

namespace rr {

hipError_t launch_route_f32_relay(const RouteArgs &a, int grid, hipStream_t stream)
{
    return route_detail::launch_family<MODE_RELAY, float>(a, grid, stream);
}

}  // namespace rr
