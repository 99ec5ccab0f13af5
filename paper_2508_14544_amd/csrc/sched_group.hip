// sched_group.hip -- the workgroup kernels (W waves per instance, ROWS
// register rows each; see k_simulate_group in sim_device.hpp), compiled on
// their own.  W x ROWS: 2 x 8 and 4 x 4 (1024 runs, for few large
// instances), 4 x 16 and 8 x 16 (4096 and 8192 runs, for the instances whose
// running set outgrows one wave).
#include "sim_device.hpp"

namespace sk {
template __global__ void k_simulate_group<SCHED_AMAX, 2, 8, false>(Params);
template __global__ void k_simulate_group<SCHED_AMAX, 4, 4, false>(Params);
template __global__ void k_simulate_group<SCHED_AMAX, 4, 16, false>(Params);
template __global__ void k_simulate_group<SCHED_AMAX, 8, 16, false>(Params);
template __global__ void k_simulate_group<SCHED_HSF, 2, 8, false>(Params);
template __global__ void k_simulate_group<SCHED_HSF, 4, 4, false>(Params);
template __global__ void k_simulate_group<SCHED_HSF, 4, 16, false>(Params);
template __global__ void k_simulate_group<SCHED_HSF, 8, 16, false>(Params);
template __global__ void k_simulate_group<SCHED_ARANDOM, 4, 16, false>(Params);
template __global__ void k_simulate_group<SCHED_ARANDOM, 8, 16, false>(Params);
template __global__ void k_simulate_group<SCHED_AELL, 4, 16, false>(Params);
template __global__ void k_simulate_group<SCHED_AELL, 8, 16, false>(Params);
template __global__ void k_simulate_group<SCHED_AMIN, 2, 8, false>(Params);
template __global__ void k_simulate_group<SCHED_AMIN, 2, 8, true>(Params);
template __global__ void k_simulate_group<SCHED_AMIN, 4, 4, false>(Params);
template __global__ void k_simulate_group<SCHED_AMIN, 4, 4, true>(Params);
template __global__ void k_simulate_group<SCHED_AMIN, 4, 16, false>(Params);
template __global__ void k_simulate_group<SCHED_AMIN, 4, 16, true>(Params);
template __global__ void k_simulate_group<SCHED_AMIN, 8, 16, true>(Params);
}  // namespace sk
