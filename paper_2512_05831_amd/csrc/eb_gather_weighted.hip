// The gather kernels with per-sample weights (a weighted sum of the bag's
// rows), instantiated apart from the unweighted ones in eb.hip.
#include "eb_gather.h"

namespace eb_gather {

KernelFn pick_weighted_kernel(bool i32, int dtype, bool team, int R, int C, bool stream, bool few,
                              bool single)
{
    return pick_kernel<true>(i32, dtype, team, R, C, stream, few, single);
}

} // namespace eb_gather
