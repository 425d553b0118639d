// Weight-gradient kernels, one column per lane (and column tiles): the launches the planner in wgrad.hip
// uses (one translation unit per layout, so the build runs in parallel).
#include "wgrad.h"

namespace psc {
namespace wg {
template hipError_t launch_wgrad<DT_F32, 8, 4, 0, false, false>(dim3, const void*, const void*, const int32_t*, const int32_t*,
                                                              const int32_t*, const WGeo&, float*, hipStream_t);
template hipError_t launch_wgrad<DT_F32, 4, 4, 0, false, false>(dim3, const void*, const void*, const int32_t*, const int32_t*,
                                                              const int32_t*, const WGeo&, float*, hipStream_t);
template hipError_t launch_wgrad<DT_F16, 8, 4, 0, false, false>(dim3, const void*, const void*, const int32_t*, const int32_t*,
                                                              const int32_t*, const WGeo&, float*, hipStream_t);
template hipError_t launch_wgrad<DT_F16, 4, 4, 0, false, false>(dim3, const void*, const void*, const int32_t*, const int32_t*,
                                                              const int32_t*, const WGeo&, float*, hipStream_t);
template hipError_t launch_wgrad<DT_F32, 8, 9, 0, false, false>(dim3, const void*, const void*, const int32_t*, const int32_t*,
                                                              const int32_t*, const WGeo&, float*, hipStream_t);
template hipError_t launch_wgrad<DT_F32, 4, 9, 0, false, false>(dim3, const void*, const void*, const int32_t*, const int32_t*,
                                                              const int32_t*, const WGeo&, float*, hipStream_t);
}  // namespace wg
}  // namespace psc
