// Instantiation of the one-row-per-lane conv kernel for fp16 storage, every
// compiled width, stride 1 and 2.
#include "conv_rows.h"

namespace psc {
namespace rw {
template hipError_t launch_rows<DT_F16, 4, 1>(const PackedView&, const ConvArgs&, const RGeo&, hipStream_t);
template hipError_t launch_rows<DT_F16, 7, 1>(const PackedView&, const ConvArgs&, const RGeo&, hipStream_t);
template hipError_t launch_rows<DT_F16, 8, 1>(const PackedView&, const ConvArgs&, const RGeo&, hipStream_t);
template hipError_t launch_rows<DT_F16, 14, 1>(const PackedView&, const ConvArgs&, const RGeo&, hipStream_t);
template hipError_t launch_rows<DT_F16, 16, 1>(const PackedView&, const ConvArgs&, const RGeo&, hipStream_t);
template hipError_t launch_rows<DT_F16, 28, 1>(const PackedView&, const ConvArgs&, const RGeo&, hipStream_t);
template hipError_t launch_rows<DT_F16, 8, 2>(const PackedView&, const ConvArgs&, const RGeo&, hipStream_t);
template hipError_t launch_rows<DT_F16, 16, 2>(const PackedView&, const ConvArgs&, const RGeo&, hipStream_t);
template hipError_t launch_rows<DT_F16, 32, 2>(const PackedView&, const ConvArgs&, const RGeo&, hipStream_t);
}  // namespace rw
}  // namespace psc
