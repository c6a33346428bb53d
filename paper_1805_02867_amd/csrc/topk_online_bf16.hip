// Top-k kernels: variant TK_ONLINE, bf16 rows (one source per instantiation
// so that the build compiles them in parallel).
#include "topk.hpp"

namespace osm {
hipError_t launch_topk_online_bf16(const TopkLaunch& a) { return launch_topk_t<bf16_t, TK_ONLINE>(a); }
}  // namespace osm
