// Instantiations of the bf16-weight matrix-core kernel with 0 hidden layer(s).
#include "mfma_bf16_impl.h"

namespace pic {
namespace mfma_bf16 {
template hipError_t launch_nh<0>(const DecodeParams &, hipStream_t, int);
}  // namespace mfma_bf16
}  // namespace pic
