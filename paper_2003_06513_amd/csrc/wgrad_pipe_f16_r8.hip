// Weight-gradient kernels, one band group per wave, chunks pipelined (f16, 8 rows per lane): launches the planner in wgrad.hip
// uses (one translation unit each, so the build runs in parallel).
#include "wgrad.h"

namespace psc {
namespace wg {
template hipError_t launch_wgrad<DT_F16, 8, 4, 0, false, true>(dim3, const void*, const void*, const int32_t*, const int32_t*,
                                                              const int32_t*, const WGeo&, float*, hipStream_t);
}  // namespace wg
}  // namespace psc
