// bf16-weight kernel family (matrix cores).  Not built yet: every shape is
// reported unsupported, so the ABI returns PIC_E_UNSUPPORTED for it.
#include "pic_internal.h"

namespace pic {

bool mfma_bf16_supports(int, int, const int32_t *) { return false; }

hipError_t launch_mfma_bf16(const DecodeParams &, hipStream_t, const char **, int *, int)
{
    return hipErrorInvalidValue;
}

}  // namespace pic
