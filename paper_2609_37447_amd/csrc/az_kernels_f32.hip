// Fused policy/value network evaluation in fp32 on the vector ALUs.
//
// One workgroup of 256 threads evaluates one board: the activations live in
// LDS as [channel][square] fp32.  Each thread owns one square and accumulates
// eight output channels at a time in registers, so every LDS read of an input
// value feeds eight FMAs; the eight weights of one (input channel, tap) are one
// contiguous, wave-uniform 32-byte load (weights packed [F/8][C][9][8]), and the
// next input channel's weights are loaded while the current ones are used.
// This is the full-precision path (AZ_F32); it is sized for small networks and
// small batches, where the network is too small to feed the matrix cores.
#include "az_internal.h"

#include <math.h>

namespace {

constexpr int NT = 256;
// LDS staging area for one convolution's weights (used when they fit), at most
// this many floats and never past the 160 KB of LDS
constexpr int WSTAGE_FLOATS = 12 * 1024;
constexpr int LDS_FLOATS = 160 * 1024 / 4;

__device__ __forceinline__ float act_fn(float y, float cap) { return fminf(fmaxf(y, 0.0f), cap); }

// out[f][sq] = act(bias[f] + sum_{c,tap} W[f][c][tap] * in[c][sq + tap] (+ out[f][sq]));
// W8 is [F/8][C][9][8]; out-of-board taps read zero.
__device__ void conv3x3_f32(const float* in, int C, const float* __restrict__ W8g,
                            const float* __restrict__ bias, float* out, int F, bool residual,
                            float cap, float* wst, int wcap) {
  const int tid = threadIdx.x, sq = tid & 63;
  // weights that fit are copied to LDS first (coalesced), so the loop below
  // reads them with LDS latency instead of L2 latency
  const float* W8 = W8g;
  if (F * C * 9 <= wcap) {
    const float4* src = reinterpret_cast<const float4*>(W8g);
    float4* dst = reinterpret_cast<float4*>(wst);
    for (int i = tid; i < F * C * 9 / 4; i += NT) dst[i] = src[i];
    __syncthreads();
    W8 = wst;
  }
  const int g = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int r = sq >> 3, c = sq & 7;
  int nb[9];
  bool ok[9];
#pragma unroll
  for (int t = 0; t < 9; ++t) {
    const int rr = r + t / 3 - 1, cc = c + t % 3 - 1;
    ok[t] = (unsigned)rr < 8u && (unsigned)cc < 8u;
    nb[t] = ok[t] ? rr * 8 + cc : sq;
  }
  for (int fb = g; fb < F / 8; fb += NT / 64) {
    const float4* w = reinterpret_cast<const float4*>(W8 + (size_t)fb * C * 72);
    float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
    float4 wc[18];
#pragma unroll
    for (int k = 0; k < 18; ++k) wc[k] = w[k];
    for (int ci = 0; ci < C; ++ci) {
      float4 wn[18];
      const float4* wnext = w + (size_t)(ci + 1 < C ? ci + 1 : ci) * 18;
#pragma unroll
      for (int k = 0; k < 18; ++k) wn[k] = wnext[k];
      const float* x = in + ci * 64;
#pragma unroll
      for (int t = 0; t < 9; ++t) {
        const float xv = ok[t] ? x[nb[t]] : 0.0f;
        const float4 a = wc[2 * t], b = wc[2 * t + 1];
        acc[0] = fmaf(a.x, xv, acc[0]);
        acc[1] = fmaf(a.y, xv, acc[1]);
        acc[2] = fmaf(a.z, xv, acc[2]);
        acc[3] = fmaf(a.w, xv, acc[3]);
        acc[4] = fmaf(b.x, xv, acc[4]);
        acc[5] = fmaf(b.y, xv, acc[5]);
        acc[6] = fmaf(b.z, xv, acc[6]);
        acc[7] = fmaf(b.w, xv, acc[7]);
      }
#pragma unroll
      for (int k = 0; k < 18; ++k) wc[k] = wn[k];
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int f = fb * 8 + j;
      float y = acc[j] + bias[f];
      if (residual) y += out[f * 64 + sq];
      out[f * 64 + sq] = act_fn(y, cap);
    }
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

// LDS: H [F][64] | X-or-T region | logits [(P+1)*64] overlapping X/T after the tower | scratch |
// weight staging
__global__ __launch_bounds__(NT) void az_net_f32_kernel(AzDevNet p, const float* __restrict__ planes,
                                                        const uint8_t* __restrict__ legal, int B,
                                                        float* __restrict__ policy,
                                                        float* __restrict__ value, int wcap) {
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
  float* wst = scratch + 16;
  const float cap = p.act_cap;

  for (int i = tid; i < Cin * 64; i += NT) Xs[i] = planes[(size_t)b * Cin * 64 + i];
  __syncthreads();

  const float* tw = static_cast<const float*>(p.tower_w);
  conv3x3_f32(Xs, Cin, static_cast<const float*>(p.stem_w), p.bias, Hs, F, false, cap, wst, wcap);
  for (int j = 0; j < p.blocks; ++j) {
    conv3x3_f32(Hs, F, tw + (size_t)(2 * j) * F * F * 9, p.bias + (size_t)(1 + 2 * j) * F, Ts, F,
                false, cap, wst, wcap);
    conv3x3_f32(Ts, F, tw + (size_t)(2 * j + 1) * F * F * 9, p.bias + (size_t)(2 + 2 * j) * F, Hs,
                F, true, cap, wst, wcap);
  }

  // heads: rows 0..P-1 policy planes, row P the value 1x1 conv; eight rows per
  // wave pass (weights [ceil((P+1)/8)][F][8]), one square per lane
  float* L = Xs;
  {
    const int sq = tid & 63, g = __builtin_amdgcn_readfirstlane(tid >> 6);
    const float4* hw = static_cast<const float4*>(p.head_w);
    for (int rb = g; rb < (P + 1 + 7) / 8; rb += NT / 64) {
      float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
      const float4* w = hw + (size_t)rb * F * 2;
      for (int f = 0; f < F; ++f) {
        const float xv = Hs[f * 64 + sq];
        const float4 a = w[2 * f], b = w[2 * f + 1];
        acc[0] = fmaf(a.x, xv, acc[0]);
        acc[1] = fmaf(a.y, xv, acc[1]);
        acc[2] = fmaf(a.z, xv, acc[2]);
        acc[3] = fmaf(a.w, xv, acc[3]);
        acc[4] = fmaf(b.x, xv, acc[4]);
        acc[5] = fmaf(b.y, xv, acc[5]);
        acc[6] = fmaf(b.z, xv, acc[6]);
        acc[7] = fmaf(b.w, xv, acc[7]);
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int row = rb * 8 + j;
        if (row <= P) L[row * 64 + sq] = acc[j] + p.head_b[row];
      }
    }
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
  const int base = F * 64 + region + 16;
  const int wcap = LDS_FLOATS - base < WSTAGE_FLOATS ? (LDS_FLOATS - base > 0 ? LDS_FLOATS - base : 0) : WSTAGE_FLOATS;
  const size_t lds = ((size_t)base + wcap) * sizeof(float);
  (void)hipGetLastError();
  if (lds > 64 * 1024) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&az_net_f32_kernel),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL(az_net_f32_kernel, dim3(B), dim3(NT), lds, s, n, planes, legal, B, policy, value, wcap);
  return hipGetLastError();
}
