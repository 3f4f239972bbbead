// Dispatch of the bf16-weight matrix-core family (kernel in mfma_bf16_impl.h;
// instantiations in k_mfma_bf16_nh{0,1,2}.hip).
#include "mfma_bf16_impl.h"

namespace pic {
namespace mfma_bf16 {

int hidden_blocks(int nl, const int32_t *widths)
{
    int m = 1;
    for (int l = 1; l < nl; ++l)
        m = widths[l] > m ? widths[l] : m;
    return (m + 15) / 16;
}

extern template hipError_t launch_nh<0>(const DecodeParams &, hipStream_t, int);
extern template hipError_t launch_nh<1>(const DecodeParams &, hipStream_t, int);
extern template hipError_t launch_nh<2>(const DecodeParams &, hipStream_t, int);

}  // namespace mfma_bf16

bool mfma_bf16_supports(int L, int nl, const int32_t *widths)
{
    return L >= 1 && L <= 12 && nl >= 2 && nl <= 4 && mfma_bf16::hidden_blocks(nl, widths) <= 4;
}

hipError_t launch_mfma_bf16(const DecodeParams &p, hipStream_t s, const char **name, int *px_per_step,
                            int num_cus)
{
    if (!p.weights_bf16 || !mfma_bf16_supports(p.L, p.nl, p.widths))
        return hipErrorInvalidValue;
    *name = "k_mfma_bf16";
    *px_per_step = 16;
    switch (p.nl - 2) {
    case 0: return mfma_bf16::launch_nh<0>(p, s, num_cus);
    case 1: return mfma_bf16::launch_nh<1>(p, s, num_cus);
    case 2: return mfma_bf16::launch_nh<2>(p, s, num_cus);
    }
    return hipErrorInvalidValue;
}

}  // namespace pic
