// Instantiations of the wide form of the tuned conv kernel (fp32 and fp16,
// 4 columns and 4 rows per lane).
#include "conv_stream.h"

namespace psc {
namespace cs {
template hipError_t launch_wide<DT_F32, 4>(const PackedView&, const ConvArgs&, const Geo&, hipStream_t);
template hipError_t launch_wide<DT_F16, 4>(const PackedView&, const ConvArgs&, const Geo&, hipStream_t);
}  // namespace cs
}  // namespace psc
