// Top-k kernels: variant TK_VALUES, bf16 rows (one source per instantiation
// so that the build compiles them in parallel).
#include "topk.hpp"

namespace osm {
hipError_t launch_topk_values_bf16(const TopkLaunch& a) { return launch_topk_t<bf16_t, TK_VALUES>(a); }
}  // namespace osm
