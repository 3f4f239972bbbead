// Instantiations of the fp32 matrix-core kernel with 1 hidden layer(s).
#include "mfma_f32_impl.h"

namespace pic {
namespace mfma_f32 {
template hipError_t launch_nh<1>(const DecodeParams &, hipStream_t, int);
}  // namespace mfma_f32
}  // namespace pic
