// Deployment validation: per-position comparison of two evaluations of the same
// positions (a test network, e.g. the quantised one, against its reference, the
// float source network), the checks the paper applies after every refit of its
// deployed engine (Section "Prediction drift under TensorRT refitting": top-one
// legal-move agreement, legal-policy KL divergence and value error).
//
// One wave per position.  Lanes stride over the cells (coalesced byte and float
// loads), keep their own legal argmax of each policy (first index on ties) and
// their part of the KL sum, and the wave combines them with shuffles.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "az.h"
#include "az_internal.h"

namespace {

constexpr int NT = 256, WPB = NT / 64;
// Probabilities of the test policy below this floor count as the floor inside
// the logarithm, so that a legal move the test network rounds to zero gives a
// large but finite KL term.
constexpr float P_FLOOR = 1e-30f;

__device__ __forceinline__ void argmax_merge(float& v, int& i, float v2, int i2) {
  if (v2 > v || (v2 == v && i2 < i)) {
    v = v2;
    i = i2;
  }
}

__global__ __launch_bounds__(NT) void az_compare_kernel(const float* __restrict__ pr,
                                                         const float* __restrict__ vr,
                                                         const float* __restrict__ pt,
                                                         const float* __restrict__ vt,
                                                         const uint8_t* __restrict__ legal, int B, int N,
                                                         float* __restrict__ out) {
  const int b = blockIdx.x * WPB + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (b >= B) return;  // the whole wave leaves together
  const size_t row = (size_t)b * N;
  float br = -1.0f, bt = -1.0f, kl = 0.0f;
  int ir = INT32_MAX, it = INT32_MAX;
  for (int i = lane; i < N; i += 64) {
    if (legal[row + i]) {
      const float a = pr[row + i], c = pt[row + i];
      if (a > br) { br = a; ir = i; }  // i increases, so the first maximum is kept
      if (c > bt) { bt = c; it = i; }
      if (a > 0.0f) kl += a * (logf(a) - logf(fmaxf(c, P_FLOOR)));
    }
  }
  for (int o = 32; o > 0; o >>= 1) {
    const float br2 = __shfl_xor(br, o), bt2 = __shfl_xor(bt, o);
    const int ir2 = __shfl_xor(ir, o), it2 = __shfl_xor(it, o);
    argmax_merge(br, ir, br2, ir2);
    argmax_merge(bt, it, bt2, it2);
    kl += __shfl_xor(kl, o);
  }
  if (lane == 0) {
    out[3 * (size_t)b] = ir == it ? 1.0f : 0.0f;  // rows without a legal move agree
    out[3 * (size_t)b + 1] = kl;
    out[3 * (size_t)b + 2] = fabsf(vr[b] - vt[b]);
  }
}

}  // namespace

extern "C" int az_compare_outputs(const float* policy_ref, const float* value_ref, const float* policy_test,
                                  const float* value_test, const uint8_t* legal, int32_t B, int32_t n_moves,
                                  float* row_metrics, void* stream) {
  if (B < 0) return az_fail(AZ_ERR_INVALID_ARG, "az_compare_outputs: B < 0");
  if (n_moves <= 0) return az_fail(AZ_ERR_INVALID_ARG, "az_compare_outputs: n_moves <= 0");
  if (B == 0) return AZ_OK;
  if (!policy_ref || !value_ref || !policy_test || !value_test || !legal || !row_metrics)
    return az_fail(AZ_ERR_INVALID_ARG, "az_compare_outputs: NULL buffer");
  if (((uintptr_t)policy_ref | (uintptr_t)value_ref | (uintptr_t)policy_test | (uintptr_t)value_test |
       (uintptr_t)row_metrics) & 3u)
    return az_fail(AZ_ERR_INVALID_ARG, "az_compare_outputs: float buffers must be 4-byte aligned");
  (void)hipGetLastError();
  hipLaunchKernelGGL(az_compare_kernel, dim3((B + WPB - 1) / WPB), dim3(NT), 0, static_cast<hipStream_t>(stream),
                     policy_ref, value_ref, policy_test, value_test, legal, B, n_moves, row_metrics);
  const hipError_t e = hipGetLastError();
  return e == hipSuccess ? AZ_OK : az_fail(AZ_ERR_DEVICE, hipGetErrorString(e));
}
