// Instantiation of the one-row-per-lane conv kernel for fp16 storage, every
// compiled width.
#include "conv_rows.h"

namespace psc {
namespace rw {
template hipError_t launch_rows<DT_F16, 4>(const PackedView&, const ConvArgs&, const RGeo&, hipStream_t);
template hipError_t launch_rows<DT_F16, 7>(const PackedView&, const ConvArgs&, const RGeo&, hipStream_t);
template hipError_t launch_rows<DT_F16, 8>(const PackedView&, const ConvArgs&, const RGeo&, hipStream_t);
template hipError_t launch_rows<DT_F16, 14>(const PackedView&, const ConvArgs&, const RGeo&, hipStream_t);
template hipError_t launch_rows<DT_F16, 16>(const PackedView&, const ConvArgs&, const RGeo&, hipStream_t);
template hipError_t launch_rows<DT_F16, 28>(const PackedView&, const ConvArgs&, const RGeo&, hipStream_t);
}  // namespace rw
}  // namespace psc
