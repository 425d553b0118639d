// Instantiation of the tuned conv kernels for fp32 storage, 7 rows per lane
// (direct, staged and multi-run staged forms).
#include "conv_stream.h"

namespace psc {
namespace cs {
template hipError_t launch_r<DT_F32, 7>(const PackedView&, const ConvArgs&, const Geo&, hipStream_t);
}  // namespace cs
}  // namespace psc
