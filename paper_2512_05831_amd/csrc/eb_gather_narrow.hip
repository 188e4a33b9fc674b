// Team gather kernels with 8- and 4-byte chunks (rows that are not a multiple
// of 16 bytes, or whose tables or output allow only narrower accesses),
// instantiated apart from the 16-byte ones so the parts build in parallel;
// the weighted ones in eb_gather_narrow_weighted.hip.
#include "eb_gather.h"

namespace eb_gather {

KernelFn pick_narrow_kernel(bool weighted, bool i32, int dtype, int cb, int R, bool stream, bool few,
                            bool single)
{
    if (weighted) return pick_narrow_weighted_kernel(i32, dtype, cb, R, stream, few, single);
    if (cb == 8) return i32 ? pick_team_kernel<int32_t, false, 8>(dtype, R, 1, stream, few, single)
                            : pick_team_kernel<int64_t, false, 8>(dtype, R, 1, stream, few, single);
    if (cb == 4) return i32 ? pick_team_kernel<int32_t, false, 4>(dtype, R, 1, stream, few, single)
                            : pick_team_kernel<int64_t, false, 4>(dtype, R, 1, stream, few, single);
    return nullptr;
}

} // namespace eb_gather
