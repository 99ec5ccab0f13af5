// sched_wide.hip -- the wide row ladder kernels (up to 16 register rows, 1024
// runs; see k_simulate_ladder_wide in sim_device.hpp), compiled on their own.
#include "sim_device.hpp"

namespace sk {
template __global__ void k_simulate_ladder_wide<SCHED_AMAX>(Params);
template __global__ void k_simulate_ladder_wide<SCHED_AMIN>(Params);
template __global__ void k_simulate_ladder_wide<SCHED_HSF>(Params);
template __global__ void k_simulate_ladder_wide<SCHED_AELL>(Params);
template __global__ void k_simulate_ladder_wide<SCHED_ARANDOM>(Params);
}  // namespace sk
