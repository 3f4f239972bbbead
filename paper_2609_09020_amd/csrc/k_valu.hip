// Dispatch of the reference kernel family (device code in valu_impl.h).  The
// instances for hidden widths up to 64 live here; the two wide ones (96 and
// 128) in k_valu_w96.hip and k_valu_w128.hip.
#include "valu_impl.h"

namespace pic {
namespace valu {
namespace {

int padded_levels(int L) { return ((L + 3) / 4) * 4; }

// Hidden widths are padded with zero neurons to a multiple of 8 up to 64, and
// to 96 or 128 above (two wide instances).
int padded_hidden(int nl, const int32_t *widths)
{
    int m = 8;
    for (int l = 1; l < nl; ++l)
        m = widths[l] > m ? widths[l] : m;
    return m <= kNarrow ? ((m + 7) / 8) * 8 : m <= 96 ? 96 : ((m + 31) / 32) * 32;
}

template <int PL>
hipError_t launch_pw(int PW, const DecodeParams &p, hipStream_t s)
{
    switch (PW) {
    case 8: return launch_t<PL, 8>(p, s);
    case 16: return launch_t<PL, 16>(p, s);
    case 24: return launch_t<PL, 24>(p, s);
    case 32: return launch_t<PL, 32>(p, s);
    case 40: return launch_t<PL, 40>(p, s);
    case 48: return launch_t<PL, 48>(p, s);
    case 56: return launch_t<PL, 56>(p, s);
    case 64: return launch_t<PL, 64>(p, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace
}  // namespace valu

bool valu_supports(int L, int nl, const int32_t *widths)
{
    return L >= 1 && L <= 12 && nl >= 1 && valu::padded_hidden(nl, widths) <= PIC_MAX_WIDTH;
}

hipError_t launch_valu(const DecodeParams &p, hipStream_t s, const char **name, int *px_per_step)
{
    if (!valu_supports(p.L, p.nl, p.widths))
        return hipErrorInvalidValue;
    const int PL = valu::padded_levels(p.L), PW = valu::padded_hidden(p.nl, p.widths);
    *px_per_step = 64;
    if (PW > valu::kNarrow) {
        *name = "k_valu_wide";
        return PW == 96 ? valu::launch_wide96(p, s) : valu::launch_wide128(p, s);
    }
    *name = "k_valu";
    switch (PL) {
    case 4: return valu::launch_pw<4>(PW, p, s);
    case 8: return valu::launch_pw<8>(PW, p, s);
    case 12: return valu::launch_pw<12>(PW, p, s);
    }
    return hipErrorInvalidValue;
}

}  // namespace pic
