// Instantiations of the fp16-split matrix-core kernel with 2 hidden layer(s).
#include "mfma_f16x3_impl.h"

namespace pic {
namespace mfma_f16x3 {
template hipError_t launch_nh<2>(const DecodeParams &, hipStream_t, int);
}  // namespace mfma_f16x3
}  // namespace pic
