// Route kernel instances: bf16 inputs, relay layers (rescoring + trigger +
// routing of the flagged rows in one pass).
#include "rr_route_impl.hpp"

namespace rr {

hipError_t launch_route_bf16_relay(const RouteArgs &a, int grid, hipStream_t stream)
{
    return route_detail::launch_family<MODE_RELAY, bf16_t>(a, grid, stream);
}

}  // namespace rr
