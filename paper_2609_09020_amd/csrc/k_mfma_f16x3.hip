// Dispatch of the fp16-split matrix-core family (kernel in
// mfma_f16x3_impl.h; the instantiations live in k_mfma_f16x3_nh{0,1,2}.hip,
// one per hidden-layer count, so they compile in parallel).
#include "mfma_f16x3_impl.h"

namespace pic {
namespace mfma_f16x3 {

int hidden_blocks(int nl, const int32_t *widths)
{
    int m = 1;
    for (int l = 1; l < nl; ++l)
        m = widths[l] > m ? widths[l] : m;
    return (m + 15) / 16;
}

int hidden_values(int nl, const int32_t *widths)
{
    int m = 1;
    for (int l = 1; l < nl; ++l)     // every hidden width: the inputs of the hidden
        m = widths[l] > m ? widths[l] : m;   // layers and of the output layer
    return (m + 3) / 4;
}

extern template hipError_t launch_nh<0>(const DecodeParams &, hipStream_t, int);
extern template hipError_t launch_nh<1>(const DecodeParams &, hipStream_t, int);
extern template hipError_t launch_nh<2>(const DecodeParams &, hipStream_t, int);

}  // namespace mfma_f16x3

bool mfma_f16x3_supports(int L, int nl, const int32_t *widths)
{
    return L >= 1 && L <= 12 && nl >= 2 && nl <= 4 && mfma_f16x3::hidden_blocks(nl, widths) <= 4;
}

hipError_t launch_mfma_f16x3(const DecodeParams &p, hipStream_t s, const char **name, int *px_per_step,
                             int num_cus)
{
    if (!mfma_f16x3_supports(p.L, p.nl, p.widths))
        return hipErrorInvalidValue;
    *name = "k_mfma_f16x3";
    *px_per_step = 16;
    switch (p.nl - 2) {
    case 0: return mfma_f16x3::launch_nh<0>(p, s, num_cus);
    case 1: return mfma_f16x3::launch_nh<1>(p, s, num_cus);
    case 2: return mfma_f16x3::launch_nh<2>(p, s, num_cus);
    }
    return hipErrorInvalidValue;
}

}  // namespace pic
