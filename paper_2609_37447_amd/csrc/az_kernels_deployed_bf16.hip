// bf16 instantiations of the deployed-network kernel (az_dep_kernel.h),
// one translation unit per element format so that they compile in parallel.
#include "az_dep_kernel.h"

hipError_t az_launch_deployed_bf16(const AzDevNet& n, int tiling, const float* planes,
                                  const uint8_t* legal, int B, float* policy, float* value, float* wdl,
                                  hipStream_t s) {
  (void)hipGetLastError();
  if (n.filters != DF || B <= 0) return hipErrorInvalidValue;
  if (tiling == 1)
    hipLaunchKernelGGL((az_dep_kernel<MK_BF16>), dim3(B), dim3(64), 0, s, n, planes, legal, policy, value, wdl);
  else if (tiling == 2)
    hipLaunchKernelGGL((az_dep_kernel4<MK_BF16>), dim3(B), dim3(256), 0, s, n, planes, legal, policy, value, wdl);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}
