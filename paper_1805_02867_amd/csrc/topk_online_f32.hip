// Top-k kernels: variant TK_ONLINE, f32 rows (one source per instantiation
// so that the build compiles them in parallel).
#include "topk.hpp"

namespace osm {
hipError_t launch_topk_online_f32(const TopkLaunch& a) { return launch_topk_t<float, TK_ONLINE>(a); }
}  // namespace osm
