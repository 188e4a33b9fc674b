// Weighted team gather kernels with 8- and 4-byte chunks (see
// eb_gather_narrow.hip), in a translation unit of their own.
#include "eb_gather.h"

namespace eb_gather {

KernelFn pick_narrow_weighted_kernel(bool i32, int dtype, int cb, int R, bool stream, bool few, bool single)
{
    if (cb == 8) return i32 ? pick_team_kernel<int32_t, true, 8>(dtype, R, 1, stream, few, single)
                            : pick_team_kernel<int64_t, true, 8>(dtype, R, 1, stream, few, single);
    if (cb == 4) return i32 ? pick_team_kernel<int32_t, true, 4>(dtype, R, 1, stream, few, single)
                            : pick_team_kernel<int64_t, true, 4>(dtype, R, 1, stream, few, single);
    return nullptr;
}

} // namespace eb_gather
