// The reference family's instance for hidden widths up to 96 (levels padded to
// 12); one translation unit of its own because it is large.
#include "valu_impl.h"

namespace pic {
namespace valu {

hipError_t launch_wide96(const DecodeParams &p, hipStream_t s) { return launch_t<12, 96>(p, s); }

}  // namespace valu
}  // namespace pic
