// int8 instantiations of the deployed-network kernel (az_dep_kernel.h),
// one translation unit per element format so that they compile in parallel.
#include "az_dep_kernel.h"

hipError_t az_launch_deployed_int8(int waves_per_board, const AzDevNet& n, const float* planes,
                                  const uint8_t* legal, int B, float* policy, float* value, float* wdl,
                                  hipStream_t s) {
  (void)hipGetLastError();
  if (n.filters != DF || B <= 0) return hipErrorInvalidValue;
  const dim3 grid(B), block(64 * waves_per_board);
  if (waves_per_board == 1)
    hipLaunchKernelGGL((az_dep_kernel<MK_I8, 1>), grid, block, 0, s, n, planes, legal, policy, value, wdl);
  else if (waves_per_board == 2)
    hipLaunchKernelGGL((az_dep_kernel<MK_I8, 2>), grid, block, 0, s, n, planes, legal, policy, value, wdl);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}
