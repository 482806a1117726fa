// sj_join_i8.hip -- instantiates the fused join kernels for I8 inputs
// (kept in its own translation unit so the element types compile in parallel).
#include "sj_join_kernels.h"

namespace sjk {

hipError_t launch_join_i8(const Plan &p, int metric, int mode, const JoinArgs &g,
                          hipStream_t st)
{
    return launch_dtype<DT_I8>(p, metric, mode, g, st);
}

int resident_occupancy_i8(int metric, int variant)
{
    return resident_occupancy_dtype<DT_I8>(metric, variant);
}

}  // namespace sjk
