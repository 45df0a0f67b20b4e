// Internal interface between the host runtime (az_runtime.cpp) and the kernels.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "az.h"

// Rows of the fused policy/value head matrix: policy planes, then the value
// 1x1 conv row, then zero rows up to three 32-row MFMA blocks.
#define AZ_HEAD_ROWS 96
// Largest policy-plane count the fused head supports (one row left for value).
#define AZ_MAX_POLICY 95
// Largest input-plane count (the stem pads its channels to 32).
#define AZ_MAX_IN_PLANES 32

// Device-side description of a loaded network, passed to kernels by value.
struct AzDevNet {
  int in_planes, blocks, filters, policy_planes, value_hidden, value_conv_relu;
  float act_cap;     // +inf when the activation is a plain ReLU
  float head_scale;  // value of one code of the final tower tensor (1 for float nets)
  // MFMA dtypes: A-fragment streams (see az_runtime.cpp for the order).
  // AZ_F32: canonical fp32 arrays.
  const void* stem_w;
  const void* tower_w;
  const void* head_w;
  // Per-channel epilogue constants, [(1 + 2*blocks) * F]: the stem, then residual
  // conv n = 0..2*blocks-1.  Float nets: bias = b.  Quantised nets, in float64:
  // the code of an output is rne(clamp(z, 0, qhi[k])) on the int8 or e4m3 grid,
  // z = acc * qmul + qbias (+ the residual and pooled terms), i.e.
  // act(y) / a[k] of the definition y = acc * a[n] * s_w[n][f] + b[f] + ...:
  //   stem:   qmul = 1/a[0],                     qbias = b / a[0]
  //   conv n: qmul = a[n] * s_w[n][f] / a[n+1],  qbias = b / a[n+1]
  const float* bias;
  const double* qmul;
  const double* qbias;
  // Quantised nets, per output tensor k = 0..2*blocks (tensor k is written by
  // conv k-1, the stem for k = 0): qres[k] = a[k-2] / a[k] for the second conv
  // of a block (its residual input's code scaled into the output's code units),
  // qhi[k] = the largest code of tensor k, min(qmax, act_cap / a[k]) rounded to
  // the code grid (activation cap and saturation).
  const double* qres;
  const float* qhi;
  // qext[2k], qext[2k + 1] = qres[k], qhi[k] (as a double): the two scalars of
  // tensor k side by side, for kernels that stage them with the per-channel ones
  const double* qext;
  const float* head_b;  // [AZ_HEAD_ROWS]: policy biases, value conv bias at row P, zeros
  const float* fc1_w;   // [H][64]
  const float* fc1_b;   // [H]
  const float* fc2_w;   // [H]
  float fc2_b;
  // MFMA kernels: per head row scale and bias (policy rows times log2(e), value
  // row P as is, zero padding) and fc1 as [64/4][H][4] (see az_runtime.cpp)
  const float* head_sc;  // [AZ_HEAD_ROWS]
  const float* head_bc;  // [AZ_HEAD_ROWS]
  const float* fc1_t;    // [16][H][4]

  // Deployed network (global pooling, from-to policy head, WDL value head); see
  // az_dep_kernel.h for the fragment orders.
  int pool_every;      // 0: no pooling blocks
  int value_channels;  // V
  const void* emb_w;   // bf16 A fragments, rows: D token rows, V value rows, zeros (AZ_DEP_EMB_ROWS)
  const void* q_w;     // bf16 A fragments of Wq, K dimension in the token accumulators' order
  const void* k_w;     // same for Wk
  const void* p_w;     // bf16 A fragments of Wp (4 rows padded to 32), K in the key accumulators' order
  const float* emb_sc;     // [AZ_DEP_EMB_ROWS] row scale (value of one unit of h)
  const float* emb_bc;     // [AZ_DEP_EMB_ROWS] row bias: be, then bv, then zeros
  const float* q_b;        // [D]
  const float* k_b;        // [D]
  const float* pool_wt;    // per pooling block (in block order): Wg as [2g/4][AZ_DEP_POOL_OPAD][4] fp32
  // int8 pooling blocks (first conv n = 2j): the pooled channels' activation is
  // act(acc * pool_m[n][f] + pool_b[n][f]) with pool_m = a[n] * s_w[n][f] and
  // pool_b = b1 (float64); the projected context c enters the regular channels'
  // requantisation as c * pool_cinv[n], pool_cinv[n] = 1 / a[n+1].
  const double* pool_m;     // [2*blocks][F]
  const double* pool_b;     // [2*blocks][F]
  const double* pool_cinv;  // [2*blocks]
  const uint32_t* actions; // [AZ_DEP_ACTION_SLOTS]: f*64 + t | (promotion c*4 + k + 1) << 12
  const float* wdl_fc1_t;  // [V*64][H] (fc1 transposed)
  const float* wdl_fc1_b;  // [H]
  const float* wdl_fc2_w;  // [3][H]
  float wdl_fc2_b[3];
};

// Deployed network constants: embedding rows (128 token rows + up to 32 value
// rows), padded pooled-projection outputs, action-table slots.
#define AZ_DEP_TOKEN 128
#define AZ_DEP_EMB_ROWS 160
#define AZ_DEP_POOL_OPAD 128
#define AZ_DEP_ACTION_SLOTS 2048
#define AZ_DEP_MAX_IN_PLANES 64

// Returns hipSuccess or the launch error.  tiling: 1 = large, 2 = small, 3 = medium.
hipError_t az_launch_mfma(int dtype, int tiling, const AzDevNet& net, const float* planes,
                          const uint8_t* legal, int B, float* policy, float* value,
                          hipStream_t stream);
// Deployed network (F = 160) in int8 or bf16; wdl may be NULL.  tiling: 1 = one
// wave per board, 2 = four waves per board.
hipError_t az_launch_deployed_int8(const AzDevNet& net, int tiling, const float* planes, const uint8_t* legal,
                                   int B, float* policy, float* value, float* wdl, hipStream_t stream);
hipError_t az_launch_deployed_bf16(const AzDevNet& net, int tiling, const float* planes, const uint8_t* legal,
                                   int B, float* policy, float* value, float* wdl, hipStream_t stream);
hipError_t az_launch_f32(const AzDevNet& net, const float* planes, const uint8_t* legal, int B,
                         float* policy, float* value, hipStream_t stream);
// Boards per workgroup of a tiling (for grid sizing and tests).
int az_mfma_boards_per_wg(int filters, int tiling);
// Whether a tiling id (1 large, 2 small, 3 medium) exists for a filter count.
bool az_mfma_tiling_valid(int filters, int tiling);
// Whether an (dtype, filters) pair has MFMA kernels in the library.
bool az_mfma_supported(int dtype, int filters);
// Device and pinned-host allocations of the library.  Every one is counted
// (az_debug_live_allocations) and can be made to fail on purpose
// (az_debug_fail_allocation) so that the failure paths can be tested.
hipError_t az_dev_malloc(void** ptr, size_t bytes);
void az_dev_free(void* ptr);
hipError_t az_host_malloc(void** ptr, size_t bytes);
void az_host_free(void* ptr);
// Records `detail` for az_last_error() and returns `status`.
int az_fail(int status, const char* detail);
// Spec (normalised to the current version) and device of a loaded handle.
const az_layer_spec& az_net_spec(const az_net* n);
// Policy entries per position of a spec: P*64, or AZ_FROMTO_ACTIONS.
int az_spec_moves(const az_layer_spec& s);
int az_net_device(const az_net* n);
