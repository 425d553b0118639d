// Weight-gradient kernels, one image row per lane (f32): launches the planner in wgrad.hip
// uses (one translation unit each, so the build runs in parallel).
#include "wgrad.h"

namespace psc {
namespace wg {
template hipError_t launch_wgrad<DT_F32, 4, 4, 4, false, false>(dim3, const void*, const void*, const int32_t*, const int32_t*,
                                                              const int32_t*, const WGeo&, float*, hipStream_t);
template hipError_t launch_wgrad<DT_F32, 4, 4, 7, false, false>(dim3, const void*, const void*, const int32_t*, const int32_t*,
                                                              const int32_t*, const WGeo&, float*, hipStream_t);
template hipError_t launch_wgrad<DT_F32, 4, 4, 8, false, false>(dim3, const void*, const void*, const int32_t*, const int32_t*,
                                                              const int32_t*, const WGeo&, float*, hipStream_t);
template hipError_t launch_wgrad<DT_F32, 4, 4, 14, false, false>(dim3, const void*, const void*, const int32_t*, const int32_t*,
                                                              const int32_t*, const WGeo&, float*, hipStream_t);
template hipError_t launch_wgrad<DT_F32, 4, 4, 16, false, false>(dim3, const void*, const void*, const int32_t*, const int32_t*,
                                                              const int32_t*, const WGeo&, float*, hipStream_t);
}  // namespace wg
}  // namespace psc
