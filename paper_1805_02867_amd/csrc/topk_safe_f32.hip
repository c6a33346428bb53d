// Top-k kernels: variant TK_SAFE, f32 rows (one source per instantiation
// so that the build compiles them in parallel).
#include "topk.hpp"

namespace osm {
hipError_t launch_topk_safe_f32(const TopkLaunch& a) { return launch_topk_t<float, TK_SAFE>(a); }
}  // namespace osm
