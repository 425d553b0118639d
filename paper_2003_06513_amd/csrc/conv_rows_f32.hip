// Instantiation of the one-row-per-lane conv kernel for fp32 storage, every
// compiled width, stride 1 and 2.
#include "conv_rows.h"

namespace psc {
namespace rw {
template hipError_t launch_rows<DT_F32, 4, 1>(const PackedView&, const ConvArgs&, const RGeo&, hipStream_t);
template hipError_t launch_rows<DT_F32, 7, 1>(const PackedView&, const ConvArgs&, const RGeo&, hipStream_t);
template hipError_t launch_rows<DT_F32, 8, 1>(const PackedView&, const ConvArgs&, const RGeo&, hipStream_t);
template hipError_t launch_rows<DT_F32, 14, 1>(const PackedView&, const ConvArgs&, const RGeo&, hipStream_t);
template hipError_t launch_rows<DT_F32, 16, 1>(const PackedView&, const ConvArgs&, const RGeo&, hipStream_t);
template hipError_t launch_rows<DT_F32, 28, 1>(const PackedView&, const ConvArgs&, const RGeo&, hipStream_t);
template hipError_t launch_rows<DT_F32, 8, 2>(const PackedView&, const ConvArgs&, const RGeo&, hipStream_t);
template hipError_t launch_rows<DT_F32, 16, 2>(const PackedView&, const ConvArgs&, const RGeo&, hipStream_t);
template hipError_t launch_rows<DT_F32, 32, 2>(const PackedView&, const ConvArgs&, const RGeo&, hipStream_t);
}  // namespace rw
}  // namespace psc
