// bf16 instantiations of the VALU route kernel.
#include "route_valu.hpp"

namespace hetumoe {

hipError_t launch_route_valu_bf16(const RouteArgs& a, hipStream_t st) { return launch_valu_dt<bf16_t>(a, st); }

}  // namespace hetumoe
