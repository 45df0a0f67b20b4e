// Fused policy/value network evaluation in fp32 on the vector ALUs.
//
// One workgroup of 256 threads evaluates one board: the activations live in
// LDS as [channel][square] fp32, every thread owns one square and a strided set
// of output channels, and weights are read with wave-uniform (scalar) loads.
// This is the full-precision path (AZ_F32); it is sized for small networks and
// small batches, where the network is too small to feed the matrix cores.
#include "az_internal.h"

#include <math.h>

namespace {

constexpr int NT = 256;

__device__ __forceinline__ float act_fn(float y, float cap) { return fminf(fmaxf(y, 0.0f), cap); }

// out[f][sq] = act(bias[f] + sum_{c,tap} W[f][c][tap] * in[c][sq + tap] (+ out[f][sq]))
__device__ void conv3x3_f32(const float* in, int C, const float* __restrict__ W,
                            const float* __restrict__ bias, float* out, int F, bool residual,
                            float cap) {
  const int tid = threadIdx.x, sq = tid & 63;
  const int fg = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r = sq >> 3, c = sq & 7;
  int nb[9];
#pragma unroll
  for (int t = 0; t < 9; ++t) {
    const int rr = r + t / 3 - 1, cc = c + t % 3 - 1;
    nb[t] = ((unsigned)rr < 8u && (unsigned)cc < 8u) ? rr * 8 + cc : -1;
  }
  for (int f = fg; f < F; f += NT / 64) {
    const float* w = W + (size_t)f * C * 9;
    float acc = 0.0f;
    for (int ci = 0; ci < C; ++ci) {
      const float* x = in + ci * 64;
#pragma unroll
      for (int t = 0; t < 9; ++t)
        if (nb[t] >= 0) acc = fmaf(w[ci * 9 + t], x[nb[t]], acc);
    }
    float y = acc + bias[f];
    if (residual) y += out[f * 64 + sq];
    out[f * 64 + sq] = act_fn(y, cap);
  }
  __syncthreads();
}

__device__ float block_reduce(float v, bool is_max, float* scratch) {
  for (int o = 32; o > 0; o >>= 1) {
    const float u = __shfl_xor(v, o);
    v = is_max ? fmaxf(v, u) : v + u;
  }
  const int tid = threadIdx.x;
  if ((tid & 63) == 0) scratch[tid >> 6] = v;
  __syncthreads();
  float r = scratch[0];
  for (int i = 1; i < NT / 64; ++i) r = is_max ? fmaxf(r, scratch[i]) : r + scratch[i];
  __syncthreads();
  return r;
}

// LDS: H [F][64] | X-or-T region | logits [(P+1)*64] overlapping X/T after the tower | scratch
__global__ __launch_bounds__(NT) void az_net_f32_kernel(AzDevNet p, const float* __restrict__ planes,
                                                        const uint8_t* __restrict__ legal, int B,
                                                        float* __restrict__ policy,
                                                        float* __restrict__ value) {
  extern __shared__ float sm[];
  const int F = p.filters, Cin = p.in_planes, P = p.policy_planes;
  const int b = blockIdx.x;
  if (b >= B) return;
  const int tid = threadIdx.x;
  float* Hs = sm;
  float* Xs = sm + F * 64;
  float* Ts = sm + F * 64 + Cin * 64;
  const int region = (Cin + F) * 64 > (P + 1) * 64 ? (Cin + F) * 64 : (P + 1) * 64;
  float* scratch = sm + F * 64 + region;
  const float cap = p.act_cap;

  for (int i = tid; i < Cin * 64; i += NT) Xs[i] = planes[(size_t)b * Cin * 64 + i];
  __syncthreads();

  const float* tw = static_cast<const float*>(p.tower_w);
  conv3x3_f32(Xs, Cin, static_cast<const float*>(p.stem_w), p.bias, Hs, F, false, cap);
  for (int j = 0; j < p.blocks; ++j) {
    conv3x3_f32(Hs, F, tw + (size_t)(2 * j) * F * F * 9, p.bias + (size_t)(1 + 2 * j) * F, Ts, F,
                false, cap);
    conv3x3_f32(Ts, F, tw + (size_t)(2 * j + 1) * F * F * 9, p.bias + (size_t)(2 + 2 * j) * F, Hs,
                F, true, cap);
  }

  // heads: rows 0..P-1 policy planes, row P the value 1x1 conv
  float* L = Xs;
  const float* hw = static_cast<const float*>(p.head_w);
  for (int i = tid; i < (P + 1) * 64; i += NT) {
    const int row = i >> 6, sq = i & 63;
    const float* wr = hw + (size_t)row * F;
    float acc = 0.0f;
    for (int f = 0; f < F; ++f) acc = fmaf(wr[f], Hs[f * 64 + sq], acc);
    L[i] = acc + p.head_b[row];
  }
  __syncthreads();

  const int NM = P * 64;
  const uint8_t* lg = legal + (size_t)b * NM;
  float* pol = policy + (size_t)b * NM;
  float mx = -INFINITY;
  for (int i = tid; i < NM; i += NT)
    if (lg[i]) mx = fmaxf(mx, L[i]);
  mx = block_reduce(mx, true, scratch);
  float sum = 0.0f;
  if (mx != -INFINITY)
    for (int i = tid; i < NM; i += NT)
      if (lg[i]) sum += expf(L[i] - mx);
  sum = block_reduce(sum, false, scratch);
  const float inv = sum > 0.0f ? 1.0f / sum : 0.0f;
  for (int i = tid; i < NM; i += NT) pol[i] = lg[i] ? expf(L[i] - mx) * inv : 0.0f;

  if (tid < 64) {
    const int lane = tid;
    const float* u = L + NM;
    float part = 0.0f;
    for (int k = lane; k < p.value_hidden; k += 64) {
      const float* wr = p.fc1_w + (size_t)k * 64;
      float g = p.fc1_b[k];
      for (int s = 0; s < 64; ++s) {
        const float us = p.value_conv_relu ? fmaxf(u[s], 0.0f) : u[s];
        g = fmaf(wr[s], us, g);
      }
      part = fmaf(p.fc2_w[k], fmaxf(g, 0.0f), part);
    }
    for (int o = 32; o > 0; o >>= 1) part += __shfl_xor(part, o);
    if (lane == 0) value[b] = tanhf(part + p.fc2_b);
  }
}

}  // namespace

hipError_t az_launch_f32(const AzDevNet& n, const float* planes, const uint8_t* legal, int B,
                         float* policy, float* value, hipStream_t s) {
  const int F = n.filters, Cin = n.in_planes, P = n.policy_planes;
  const int region = (Cin + F) * 64 > (P + 1) * 64 ? (Cin + F) * 64 : (P + 1) * 64;
  const size_t lds = ((size_t)F * 64 + region + 16) * sizeof(float);
  (void)hipGetLastError();
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&az_net_f32_kernel),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(az_net_f32_kernel, dim3(B), dim3(NT), lds, s, n, planes, legal, B, policy, value);
  return hipGetLastError();
}
