// fp32 instantiations of the VALU route kernel (also used when logits are given).
#include "route_valu.hpp"

namespace hetumoe {

hipError_t launch_route_valu_f32(const RouteArgs& a, hipStream_t st) { return launch_valu_dt<float>(a, st); }

}  // namespace hetumoe
