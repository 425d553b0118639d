// Instantiation of the wide form of the tuned conv kernel (fp32, 4 columns
// and 4 rows per lane).
#include "conv_stream.h"

namespace psc {
namespace cs {
template hipError_t launch_wide<4>(const PackedView&, const ConvArgs&, const Geo&, hipStream_t);
}  // namespace cs
}  // namespace psc
