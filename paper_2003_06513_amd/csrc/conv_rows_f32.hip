// Instantiation of the one-row-per-lane conv kernel for fp32 storage, every
// compiled width.
#include "conv_rows.h"

namespace psc {
namespace rw {
template hipError_t launch_rows<DT_F32, 4>(const PackedView&, const ConvArgs&, const RGeo&, hipStream_t);
template hipError_t launch_rows<DT_F32, 7>(const PackedView&, const ConvArgs&, const RGeo&, hipStream_t);
template hipError_t launch_rows<DT_F32, 8>(const PackedView&, const ConvArgs&, const RGeo&, hipStream_t);
template hipError_t launch_rows<DT_F32, 14>(const PackedView&, const ConvArgs&, const RGeo&, hipStream_t);
template hipError_t launch_rows<DT_F32, 16>(const PackedView&, const ConvArgs&, const RGeo&, hipStream_t);
template hipError_t launch_rows<DT_F32, 28>(const PackedView&, const ConvArgs&, const RGeo&, hipStream_t);
}  // namespace rw
}  // namespace psc
