// Weight-gradient kernels, four columns per lane: the launches the planner in wgrad.hip
// uses (one translation unit per layout, so the build runs in parallel).
#include "wgrad.h"

namespace psc {
namespace wg {
template hipError_t launch_wgrad<DT_F32, kWideRows, 4, 0, true, false>(dim3, const void*, const void*, const int32_t*, const int32_t*,
                                                              const int32_t*, const WGeo&, float*, hipStream_t);
template hipError_t launch_wgrad<DT_F16, kWideRows, 4, 0, true, false>(dim3, const void*, const void*, const int32_t*, const int32_t*,
                                                              const int32_t*, const WGeo&, float*, hipStream_t);
template hipError_t launch_wgrad<DT_F32, kWideRows, 9, 0, true, false>(dim3, const void*, const void*, const int32_t*, const int32_t*,
                                                              const int32_t*, const WGeo&, float*, hipStream_t);
}  // namespace wg
}  // namespace psc
