// Fused policy/value network evaluation on CDNA4 matrix cores (gfx950).
//
// One kernel evaluates the whole network for a tile of boards: stem, every
// residual block, the policy and value heads, the legal-move softmax and the
// tanh value.  Activations never leave the workgroup's LDS; the only HBM
// traffic is the input planes, the legal mask, the outputs and the weight
// stream (which stays resident in L2 / the Infinity Cache across workgroups).
//
// Every 3x3 convolution is an implicit GEMM per board:
//   D[ch][sq] = sum_k W[ch][k] * X[k][sq],  k = tap * C_in + c,
//   X[tap*C_in + c][sq] = act[c][sq shifted by tap]   (zero outside the board)
// with output channels as the MFMA M dimension (A operand = weights, streamed
// from global memory in pre-packed fragment order) and board squares as the N
// dimension (B operand = activations, read from LDS).  A 32x32 MFMA block
// covers 32 channels x 32 squares (half a board).  The tap loop is the K loop:
// no im2col is materialised; a shifted window is just a different LDS row per
// lane, and out-of-board taps read a zero row.
//
// Activation layout in LDS: [board][square][channel], one row of F channels
// per square, stored in 16-byte chunks whose position is XOR-swizzled by the
// square index so that the 16 lanes of a ds_read_b128 group (16 consecutive
// squares, same logical chunk) hit 16 different bank groups.
//
// MFMA output layout (32x32 blocks): lane l holds column l%32 and rows
// 8*(v/4) + 4*(l/32) + v%4 of its 16 accumulators v, i.e. four runs of four
// consecutive channels of one square, which the epilogue packs and stores with
// one LDS write per run.
#include "az_internal.h"

#include <math.h>

namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) int i32x4;
typedef __attribute__((ext_vector_type(8))) int i32x8;
typedef __attribute__((ext_vector_type(16))) int i32x16;

enum { MK_BF16 = 0, MK_I8 = 1, MK_F8 = 2 };

template <int MK> struct Mk;
template <> struct Mk<MK_BF16> {
  static constexpr int KS = 16;  // reduction length of one instruction
  static constexpr int FB = 16;  // operand bytes per lane
  static constexpr int ES = 2;   // activation element bytes
  using frag = bf16x8;
  using acc = f32x16;
  static __device__ __forceinline__ acc mma(const frag& a, const frag& b, const acc& c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
  }
};
template <> struct Mk<MK_I8> {
  static constexpr int KS = 32, FB = 16, ES = 1;
  using frag = i32x4;
  using acc = i32x16;
  static __device__ __forceinline__ acc mma(const frag& a, const frag& b, const acc& c) {
    return __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, c, 0, 0, 0);
  }
};
template <> struct Mk<MK_F8> {
  static constexpr int KS = 64, FB = 32, ES = 1;
  using frag = i32x8;
  using acc = f32x16;
  static __device__ __forceinline__ acc mma(const frag& a, const frag& b, const acc& c) {
    // Format selectors 0/0 = e4m3 for both operands; zero scales select the
    // unscaled instruction.
    return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, 0, 0, 0, 0);
  }
};

constexpr int cmax(int a, int b) { return a > b ? a : b; }

// Chunk swizzle for a row of RB bytes: rows of 256 bytes or more XOR with the
// low four square bits; shorter rows first spread consecutive squares over the
// bank groups a 256-byte line offers.
template <int RB>
__device__ __forceinline__ int swz(int sq) {
  if constexpr (RB >= 256) return sq & 15;
  else if constexpr (RB == 128) return (sq >> 1) & 7;
  else {
    static_assert(RB == 64, "row size");
    return (sq >> 2) & 3;
  }
}

template <int MK>
__device__ __forceinline__ typename Mk<MK>::frag lds_frag(const uint8_t* smem, int row, int sw, int lc) {
  if constexpr (MK == MK_F8) {
    const i32x4 lo = *reinterpret_cast<const i32x4*>(smem + row + ((lc ^ sw) << 4));
    const i32x4 hi = *reinterpret_cast<const i32x4*>(smem + row + (((lc + 1) ^ sw) << 4));
    return i32x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  } else {
    return *reinterpret_cast<const typename Mk<MK>::frag*>(smem + row + ((lc ^ sw) << 4));
  }
}

template <int MK>
__device__ __forceinline__ typename Mk<MK>::frag g_frag(const uint8_t* p) {
  return *reinterpret_cast<const typename Mk<MK>::frag*>(p);
}

__device__ __forceinline__ uint32_t bf16_bits(float f) {
  return (uint32_t)__builtin_bit_cast(unsigned short, (__bf16)f);
}
__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  return bf16_bits(a) | (bf16_bits(b) << 16);
}
__device__ __forceinline__ float bf16_lo(uint32_t x) { return __uint_as_float(x << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t x) { return __uint_as_float(x & 0xffff0000u); }

__device__ __forceinline__ float act_fn(float y, float cap) { return fminf(fmaxf(y, 0.0f), cap); }

__device__ __forceinline__ uint32_t q_i8(float v) {
  v = fminf(fmaxf(rintf(v), -127.0f), 127.0f);
  return (uint32_t)((int)v) & 0xffu;
}
__device__ __forceinline__ uint32_t pack_q4(int mk, float y0, float y1, float y2, float y3) {
  if (mk == MK_I8) return q_i8(y0) | (q_i8(y1) << 8) | (q_i8(y2) << 16) | (q_i8(y3) << 24);
  // The hardware conversion rounds to nearest even but turns |x| > 448 into
  // NaN, so saturate first.
  y0 = fminf(fmaxf(y0, -448.0f), 448.0f);
  y1 = fminf(fmaxf(y1, -448.0f), 448.0f);
  y2 = fminf(fmaxf(y2, -448.0f), 448.0f);
  y3 = fminf(fmaxf(y3, -448.0f), 448.0f);
  int w = __builtin_amdgcn_cvt_pk_fp8_f32(y0, y1, 0, false);
  w = __builtin_amdgcn_cvt_pk_fp8_f32(y2, y3, w, true);
  return (uint32_t)w;
}
template <int R>
__device__ __forceinline__ float dq_code(int mk, uint32_t x) {
  if (mk == MK_I8) return (float)(int)(int8_t)(x >> (8 * R));
  return __builtin_amdgcn_cvt_f32_fp8((int)x, R);
}

__device__ __forceinline__ float wave_max(float v) {
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// Per-tap LDS row addresses of the wave's N-blocks (square = half a board).
template <int RB_IN, int NBW>
__device__ __forceinline__ void tap_rows(int tap, int in_off, int zero_off, int nb0, int l32,
                                         int (&row)[NBW], int (&sw)[NBW]) {
  const int dy = tap / 3 - 1, dx = tap % 3 - 1;
#pragma unroll
  for (int i = 0; i < NBW; ++i) {
    const int nb = nb0 + i, bl = nb >> 1, j = ((nb & 1) << 5) + l32;
    const int r = (j >> 3) + dy, c = (j & 7) + dx;
    const bool ok = (unsigned)r < 8u && (unsigned)c < 8u;
    const int src = r * 8 + c;
    row[i] = ok ? in_off + (bl * 64 + src) * RB_IN : zero_off;
    sw[i] = ok ? swz<RB_IN>(src) : 0;
  }
}

// Tile shape: the wave owns MBW 32-channel blocks x NBW 32-square blocks; the
// workgroup is WM x WN waves; G consecutive K steps form one prefetch group.
template <int MK, int F, int MBW, int NBW, int WM, int WN, int G>
struct Cfg {
  using T = Mk<MK>;
  static constexpr int NW = WM * WN, NT = 64 * NW;
  static constexpr int BPW = NBW * WN / 2;  // boards per workgroup
  static constexpr int NMB = F / 32;
  static_assert(NMB == MBW * WM, "channel tiling");
  static_assert(NBW % 2 == 0 || WN == 1, "board tiling");
  static constexpr int RB = F * T::ES;  // bytes per square row, tower tensors
  static constexpr int BUF = BPW * 64 * RB;
  static constexpr int OFF_H = 0, OFF_T = BUF, OFF_Z = 2 * BUF;
  static constexpr int ZB = cmax(RB, 64);
  static constexpr int RBX = 2 * F;  // bf16 row bytes of the heads' input
  static constexpr int OFF_X = MK == MK_BF16 ? OFF_H : OFF_T;
  static constexpr int LBMAX = (AZ_MAX_POLICY + 1) * 64;  // floats per board, logits + u
  static constexpr int SMEM =
      cmax(cmax(2 * BUF + ZB, OFF_X + BPW * 64 * RBX), BPW * LBMAX * 4);
  static_assert(SMEM <= 160 * 1024, "LDS");
  static constexpr int CPT = F / T::KS;  // K steps per tap
  static_assert(CPT % G == 0, "group size");
  static constexpr int GPT = CPT / G, GPL = 9 * GPT;
  static constexpr int STEP_BYTES = NMB * 64 * T::FB;
  static constexpr size_t LAYER_BYTES = (size_t)9 * CPT * STEP_BYTES;
  static constexpr int NBH = (2 * BPW + NW - 1) / NW;  // head N-blocks per wave
};

template <int MK, int F, int MBW, int NBW, int WM, int WN, int G>
__global__ __launch_bounds__(64 * WM * WN, 1) void az_net_kernel(
    AzDevNet p, const float* __restrict__ planes, const uint8_t* __restrict__ legal, int B,
    float* __restrict__ policy, float* __restrict__ value) {
  using C = Cfg<MK, F, MBW, NBW, WM, WN, G>;
  using T = typename C::T;
  using SB = Mk<MK_BF16>;
  using frag_t = typename T::frag;
  using acc_t = typename T::acc;
  constexpr int NW = C::NW, NT = C::NT, BPW = C::BPW, NMB = C::NMB, RB = C::RB;
  constexpr int OFF_H = C::OFF_H, OFF_T = C::OFF_T, OFF_Z = C::OFF_Z;

  __shared__ __attribute__((aligned(16))) uint8_t smem[C::SMEM];

  const int tid = threadIdx.x, lane = tid & 63;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = w % WM, wn = w / WM;
  const int l32 = lane & 31, lhi = lane >> 5;
  const int mb0 = wm * MBW, nb0 = wn * NBW;
  const int b0 = blockIdx.x * BPW;
  const int Cin = p.in_planes;
  const float cap = p.act_cap;

  // ---- ingest: zero row, planes -> bf16 [board][square][32 channels] at OFF_T
  for (int i = tid; i < C::ZB / 16; i += NT)
    *reinterpret_cast<i32x4*>(smem + OFF_Z + i * 16) = i32x4{0, 0, 0, 0};
  for (int idx = tid; idx < BPW * 256; idx += NT) {
    const int sq = idx & 63, ck = (idx >> 6) & 3, bl = idx >> 8, b = b0 + bl;
    uint32_t pk[4];
#pragma unroll
    for (int t = 0; t < 8; t += 2) {
      const int c = ck * 8 + t;
      const float v0 = (b < B && c < Cin) ? planes[((size_t)b * Cin + c) * 64 + sq] : 0.0f;
      const float v1 = (b < B && c + 1 < Cin) ? planes[((size_t)b * Cin + c + 1) * 64 + sq] : 0.0f;
      pk[t / 2] = pack_bf16x2(v0, v1);
    }
    *reinterpret_cast<i32x4*>(smem + OFF_T + (bl * 64 + sq) * 64 + ((ck ^ swz<64>(sq)) << 4)) =
        i32x4{(int)pk[0], (int)pk[1], (int)pk[2], (int)pk[3]};
  }
  __syncthreads();

  // ---- stem: bf16 3x3 conv over 32 (padded) input channels, K = 288
  {
    constexpr int SSTEP = NMB * 64 * 16;
    const uint8_t* sw8 = static_cast<const uint8_t*>(p.stem_w) + (size_t)(mb0 * 64 + lane) * 16;
    f32x16 sacc[MBW][NBW];
#pragma unroll
    for (int m = 0; m < MBW; ++m)
#pragma unroll
      for (int n = 0; n < NBW; ++n) sacc[m][n] = f32x16{};
    SB::frag a[2][2][MBW];
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
      for (int m = 0; m < MBW; ++m) a[0][s][m] = g_frag<MK_BF16>(sw8 + s * SSTEP + m * 64 * 16);
    int row[NBW], sw[NBW];
#pragma unroll
    for (int tap = 0; tap < 9; ++tap) {
      if (tap + 1 < 9) {
#pragma unroll
        for (int s = 0; s < 2; ++s)
#pragma unroll
          for (int m = 0; m < MBW; ++m)
            a[(tap + 1) & 1][s][m] =
                g_frag<MK_BF16>(sw8 + ((tap + 1) * 2 + s) * SSTEP + m * 64 * 16);
      }
      tap_rows<64, NBW>(tap, OFF_T, OFF_Z, nb0, l32, row, sw);
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        SB::frag bfr[NBW];
#pragma unroll
        for (int n = 0; n < NBW; ++n) bfr[n] = lds_frag<MK_BF16>(smem, row[n], sw[n], 2 * s + lhi);
#pragma unroll
        for (int m = 0; m < MBW; ++m)
#pragma unroll
          for (int n = 0; n < NBW; ++n) sacc[m][n] = SB::mma(a[tap & 1][s][m], bfr[n], sacc[m][n]);
      }
    }
    // epilogue: bias, activation, store in the tower format at OFF_H
    {
#pragma clang fp contract(off)
      const float inv0 = MK == MK_BF16 ? 1.0f : p.inv[0];
#pragma unroll
      for (int m = 0; m < MBW; ++m)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int ch0 = (mb0 + m) * 32 + 8 * q + 4 * lhi;
          const float4 bb = *reinterpret_cast<const float4*>(p.bias + ch0);
#pragma unroll
          for (int n = 0; n < NBW; ++n) {
            const int nb = nb0 + n, bl = nb >> 1, j = ((nb & 1) << 5) + l32;
            const f32x16& v = sacc[m][n];
            const float y0 = act_fn(v[4 * q + 0] + bb.x, cap), y1 = act_fn(v[4 * q + 1] + bb.y, cap);
            const float y2 = act_fn(v[4 * q + 2] + bb.z, cap), y3 = act_fn(v[4 * q + 3] + bb.w, cap);
            const int rowo = OFF_H + (bl * 64 + j) * RB;
            if constexpr (MK == MK_BF16) {
              *reinterpret_cast<uint2*>(smem + rowo + (((ch0 >> 3) ^ swz<RB>(j)) << 4) + 8 * lhi) =
                  make_uint2(pack_bf16x2(y0, y1), pack_bf16x2(y2, y3));
            } else {
              *reinterpret_cast<uint32_t*>(smem + rowo + (((ch0 >> 4) ^ swz<RB>(j)) << 4) + (ch0 & 15)) =
                  pack_q4(MK, y0 * inv0, y1 * inv0, y2 * inv0, y3 * inv0);
            }
          }
        }
    }
  }
  __syncthreads();

  // ---- residual tower: 2*blocks convolutions, H -> T -> H ...
  {
    constexpr int GPL = C::GPL, GPT = C::GPT;
    const int NG = 2 * p.blocks * GPL;
    const uint8_t* tw = static_cast<const uint8_t*>(p.tower_w) + (size_t)(mb0 * 64 + lane) * T::FB;
    frag_t A0[G][MBW], A1[G][MBW];
    acc_t c[MBW][NBW];
#pragma unroll
    for (int m = 0; m < MBW; ++m)
#pragma unroll
      for (int n = 0; n < NBW; ++n) c[m][n] = acc_t{};
    int row[NBW], sw[NBW];

    auto load = [&](frag_t(&dst)[G][MBW], int g) {
      const int layer = g / GPL, gi = g - layer * GPL;
      const uint8_t* src = tw + layer * C::LAYER_BYTES + (size_t)gi * G * C::STEP_BYTES;
#pragma unroll
      for (int s = 0; s < G; ++s)
#pragma unroll
        for (int m = 0; m < MBW; ++m) dst[s][m] = g_frag<MK>(src + s * C::STEP_BYTES + m * 64 * T::FB);
    };

    auto epilogue = [&](int n_conv) {
#pragma clang fp contract(off)
      const bool second = n_conv & 1;
      const int out_off = second ? OFF_H : OFF_T;
      const float* bias = p.bias + (size_t)(1 + n_conv) * F;
      float inv_out = 1.0f, a_res = 0.0f;
      const float* ms = nullptr;
      if constexpr (MK != MK_BF16) {
        inv_out = p.inv[n_conv + 1];
        a_res = second ? p.act[n_conv - 1] : 0.0f;
        ms = p.mscale + (size_t)n_conv * F;
      }
#pragma unroll
      for (int m = 0; m < MBW; ++m)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int ch0 = (mb0 + m) * 32 + 8 * q + 4 * lhi;
          const float4 bb = *reinterpret_cast<const float4*>(bias + ch0);
          float4 mm = make_float4(1.f, 1.f, 1.f, 1.f);
          if constexpr (MK != MK_BF16) mm = *reinterpret_cast<const float4*>(ms + ch0);
#pragma unroll
          for (int n = 0; n < NBW; ++n) {
            const int nb = nb0 + n, bl = nb >> 1, j = ((nb & 1) << 5) + l32;
            const int rowo = out_off + (bl * 64 + j) * RB;
            const acc_t& v = c[m][n];
            if constexpr (MK == MK_BF16) {
              const int addr = rowo + (((ch0 >> 3) ^ swz<RB>(j)) << 4) + 8 * lhi;
              float y0 = v[4 * q + 0] + bb.x, y1 = v[4 * q + 1] + bb.y;
              float y2 = v[4 * q + 2] + bb.z, y3 = v[4 * q + 3] + bb.w;
              if (second) {
                const uint2 r = *reinterpret_cast<const uint2*>(smem + addr);
                y0 = y0 + bf16_lo(r.x);
                y1 = y1 + bf16_hi(r.x);
                y2 = y2 + bf16_lo(r.y);
                y3 = y3 + bf16_hi(r.y);
              }
              *reinterpret_cast<uint2*>(smem + addr) =
                  make_uint2(pack_bf16x2(act_fn(y0, cap), act_fn(y1, cap)),
                             pack_bf16x2(act_fn(y2, cap), act_fn(y3, cap)));
            } else {
              const int addr = rowo + (((ch0 >> 4) ^ swz<RB>(j)) << 4) + (ch0 & 15);
              float y0 = (float)v[4 * q + 0] * mm.x, y1 = (float)v[4 * q + 1] * mm.y;
              float y2 = (float)v[4 * q + 2] * mm.z, y3 = (float)v[4 * q + 3] * mm.w;
              y0 = y0 + bb.x;
              y1 = y1 + bb.y;
              y2 = y2 + bb.z;
              y3 = y3 + bb.w;
              if (second) {
                const uint32_t r = *reinterpret_cast<const uint32_t*>(smem + addr);
                y0 = y0 + dq_code<0>(MK, r) * a_res;
                y1 = y1 + dq_code<1>(MK, r) * a_res;
                y2 = y2 + dq_code<2>(MK, r) * a_res;
                y3 = y3 + dq_code<3>(MK, r) * a_res;
              }
              *reinterpret_cast<uint32_t*>(smem + addr) =
                  pack_q4(MK, act_fn(y0, cap) * inv_out, act_fn(y1, cap) * inv_out,
                          act_fn(y2, cap) * inv_out, act_fn(y3, cap) * inv_out);
            }
          }
        }
    };

    auto body = [&](int g, frag_t(&cur)[G][MBW], frag_t(&nxt)[G][MBW]) {
      if (g + 1 < NG) load(nxt, g + 1);
      const int layer = g / GPL, gi = g - layer * GPL, tap = gi / GPT, gs = gi - tap * GPT;
      const int in_off = (layer & 1) ? OFF_T : OFF_H;
      if (gs == 0) tap_rows<RB, NBW>(tap, in_off, OFF_Z, nb0, l32, row, sw);
#pragma unroll
      for (int s = 0; s < G; ++s) {
        const int cs = gs * G + s;
        const int lc = MK == MK_F8 ? 4 * cs + 2 * lhi : 2 * cs + lhi;
        frag_t bfr[NBW];
#pragma unroll
        for (int n = 0; n < NBW; ++n) bfr[n] = lds_frag<MK>(smem, row[n], sw[n], lc);
#pragma unroll
        for (int m = 0; m < MBW; ++m)
#pragma unroll
          for (int n = 0; n < NBW; ++n) c[m][n] = T::mma(cur[s][m], bfr[n], c[m][n]);
      }
      if (gi == GPL - 1) {
        epilogue(layer);
        __syncthreads();
#pragma unroll
        for (int m = 0; m < MBW; ++m)
#pragma unroll
          for (int n = 0; n < NBW; ++n) c[m][n] = acc_t{};
      }
    };

    load(A0, 0);
    for (int g = 0; g < NG; g += 2) {
      body(g, A0, A1);
      body(g + 1, A1, A0);
    }
  }

  // ---- heads: 1x1 convs F -> (P policy planes + 1 value row) as one bf16 GEMM
  const int P = p.policy_planes;
  const int LB = (P + 1) * 64;
  {
    constexpr int HS = F / 16, RBX = C::RBX, OFF_X = C::OFF_X, NBH = C::NBH;
    SB::frag ha[HS][3];
    const uint8_t* hw = static_cast<const uint8_t*>(p.head_w) + (size_t)lane * 16;
#pragma unroll
    for (int s = 0; s < HS; ++s)
#pragma unroll
      for (int m = 0; m < 3; ++m) ha[s][m] = g_frag<MK_BF16>(hw + ((s * 3 + m) * 64) * 16);

    if constexpr (MK != MK_BF16) {
      // codes -> exact bf16 values (int8 and e4m3 values are bf16-representable)
      for (int idx = tid; idx < BPW * 64 * (F / 8); idx += NT) {
        const int k = idx % (F / 8), sq = (idx / (F / 8)) & 63, bl = idx / (64 * (F / 8));
        const uint2 v = *reinterpret_cast<const uint2*>(
            smem + OFF_H + (bl * 64 + sq) * RB + (((k >> 1) ^ swz<RB>(sq)) << 4) + (k & 1) * 8);
        const uint4 o = make_uint4(pack_bf16x2(dq_code<0>(MK, v.x), dq_code<1>(MK, v.x)),
                                   pack_bf16x2(dq_code<2>(MK, v.x), dq_code<3>(MK, v.x)),
                                   pack_bf16x2(dq_code<0>(MK, v.y), dq_code<1>(MK, v.y)),
                                   pack_bf16x2(dq_code<2>(MK, v.y), dq_code<3>(MK, v.y)));
        *reinterpret_cast<uint4*>(smem + OFF_X + (bl * 64 + sq) * RBX + ((k ^ swz<RBX>(sq)) << 4)) = o;
      }
      __syncthreads();
    }

    f32x16 hacc[NBH][3];
#pragma unroll
    for (int k = 0; k < NBH; ++k) {
#pragma unroll
      for (int m = 0; m < 3; ++m) hacc[k][m] = f32x16{};
      const int nb = w + k * NW;
      if (nb < 2 * BPW) {
        const int bl = nb >> 1, j = ((nb & 1) << 5) + l32;
        const int rowx = OFF_X + (bl * 64 + j) * RBX, swx = swz<RBX>(j);
#pragma unroll
        for (int s = 0; s < HS; ++s) {
          const SB::frag bfr = lds_frag<MK_BF16>(smem, rowx, swx, 2 * s + lhi);
#pragma unroll
          for (int m = 0; m < 3; ++m) hacc[k][m] = SB::mma(ha[s][m], bfr, hacc[k][m]);
        }
      }
    }
    __syncthreads();
    float* L = reinterpret_cast<float*>(smem);
    const float hs = p.head_scale;
#pragma unroll
    for (int k = 0; k < NBH; ++k) {
      const int nb = w + k * NW;
      if (nb < 2 * BPW) {
        const int bl = nb >> 1, j = ((nb & 1) << 5) + l32;
#pragma unroll
        for (int m = 0; m < 3; ++m)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int i = m * 32 + 8 * (v >> 2) + 4 * lhi + (v & 3);
            if (i <= P) L[bl * LB + i * 64 + j] = hacc[k][m][v] * hs + p.head_b[i];
          }
      }
    }
  }
  __syncthreads();

  // ---- legal-move softmax and value head: one wave per board
  {
    const float* L = reinterpret_cast<const float*>(smem);
    const int NM = P * 64, n16 = NM >> 4, H = p.value_hidden;
    constexpr int NCH = (AZ_MAX_POLICY * 4 + 63) / 64;
    for (int bl = w; bl < BPW; bl += NW) {
      const int b = b0 + bl;
      if (b >= B) continue;
      const float* Lb = L + bl * LB;
      const uint8_t* lg = legal + (size_t)b * NM;
      float* pol = policy + (size_t)b * NM;
      uint4 mk[NCH];
      float mx = -INFINITY;
#pragma unroll
      for (int i = 0; i < NCH; ++i) {
        const int ch = lane + 64 * i;
        mk[i] = make_uint4(0, 0, 0, 0);
        if (ch < n16) {
          mk[i] = *reinterpret_cast<const uint4*>(lg + ch * 16);
          const uint32_t wd[4] = {mk[i].x, mk[i].y, mk[i].z, mk[i].w};
#pragma unroll
          for (int t = 0; t < 16; ++t)
            if ((wd[t >> 2] >> (8 * (t & 3))) & 0xffu) mx = fmaxf(mx, Lb[ch * 16 + t]);
        }
      }
      mx = wave_max(mx);
      float sum = 0.0f;
      if (mx != -INFINITY) {
#pragma unroll
        for (int i = 0; i < NCH; ++i) {
          const int ch = lane + 64 * i;
          if (ch < n16) {
            const uint32_t wd[4] = {mk[i].x, mk[i].y, mk[i].z, mk[i].w};
#pragma unroll
            for (int t = 0; t < 16; ++t)
              if ((wd[t >> 2] >> (8 * (t & 3))) & 0xffu) sum += expf(Lb[ch * 16 + t] - mx);
          }
        }
      }
      sum = wave_sum(sum);
      const float inv = sum > 0.0f ? 1.0f / sum : 0.0f;
#pragma unroll
      for (int i = 0; i < NCH; ++i) {
        const int ch = lane + 64 * i;
        if (ch < n16) {
          const uint32_t wd[4] = {mk[i].x, mk[i].y, mk[i].z, mk[i].w};
          float o[16];
#pragma unroll
          for (int t = 0; t < 16; ++t)
            o[t] = ((wd[t >> 2] >> (8 * (t & 3))) & 0xffu) ? expf(Lb[ch * 16 + t] - mx) * inv : 0.0f;
          float4* dst = reinterpret_cast<float4*>(pol + ch * 16);
          dst[0] = make_float4(o[0], o[1], o[2], o[3]);
          dst[1] = make_float4(o[4], o[5], o[6], o[7]);
          dst[2] = make_float4(o[8], o[9], o[10], o[11]);
          dst[3] = make_float4(o[12], o[13], o[14], o[15]);
        }
      }
      // value: u (64 squares) -> FC H -> ReLU -> FC 1 -> tanh
      float u[64];
#pragma unroll
      for (int s = 0; s < 64; s += 4) {
        const float4 t4 = *reinterpret_cast<const float4*>(Lb + NM + s);
        u[s] = t4.x; u[s + 1] = t4.y; u[s + 2] = t4.z; u[s + 3] = t4.w;
      }
      if (p.value_conv_relu) {
#pragma unroll
        for (int s = 0; s < 64; ++s) u[s] = fmaxf(u[s], 0.0f);
      }
      float part = 0.0f;
      for (int k = lane; k < H; k += 64) {
        const float4* wr = reinterpret_cast<const float4*>(p.fc1_w + (size_t)k * 64);
        float g = p.fc1_b[k];
#pragma unroll
        for (int s = 0; s < 16; ++s) {
          const float4 ww = wr[s];
          g += ww.x * u[4 * s] + ww.y * u[4 * s + 1] + ww.z * u[4 * s + 2] + ww.w * u[4 * s + 3];
        }
        part += p.fc2_w[k] * fmaxf(g, 0.0f);
      }
      part = wave_sum(part);
      if (lane == 0) value[b] = tanhf(part + p.fc2_b);
    }
  }
}

template <int MK, int F, int MBW, int NBW, int WM, int WN, int G>
hipError_t launch_cfg(const AzDevNet& n, const float* planes, const uint8_t* legal, int B,
                      float* policy, float* value, hipStream_t s) {
  using C = Cfg<MK, F, MBW, NBW, WM, WN, G>;
  const int grid = (B + C::BPW - 1) / C::BPW;
  hipLaunchKernelGGL((az_net_kernel<MK, F, MBW, NBW, WM, WN, G>), dim3(grid), dim3(C::NT), 0, s, n,
                     planes, legal, B, policy, value);
  return hipGetLastError();
}

// Tilings.  Large: four boards per workgroup (two for F = 256), each wave a
// 64-channel x 2-board tile.  Small: one board per workgroup.
template <int MK, int F>
hipError_t launch_f(int tiling, const AzDevNet& n, const float* planes, const uint8_t* legal, int B,
                    float* policy, float* value, hipStream_t s) {
  constexpr int CPT = F / Mk<MK>::KS;
  constexpr int G = CPT < 8 ? CPT : 8;
  if constexpr (F == 128) {
    if (tiling == 1) return launch_cfg<MK, 128, 2, 4, 2, 2, G>(n, planes, legal, B, policy, value, s);
    return launch_cfg<MK, 128, 1, 2, 4, 1, G>(n, planes, legal, B, policy, value, s);
  } else if constexpr (F == 256) {
    if (tiling == 1) return launch_cfg<MK, 256, 2, 4, 4, 1, G>(n, planes, legal, B, policy, value, s);
    return launch_cfg<MK, 256, 2, 2, 4, 1, G>(n, planes, legal, B, policy, value, s);
  } else {
    static_assert(F == 64, "filters");
    if (tiling == 1) return launch_cfg<MK, 64, 1, 4, 2, 2, G>(n, planes, legal, B, policy, value, s);
    return launch_cfg<MK, 64, 1, 2, 2, 1, G>(n, planes, legal, B, policy, value, s);
  }
}

template <int MK>
hipError_t launch_mk(int tiling, const AzDevNet& n, const float* planes, const uint8_t* legal, int B,
                     float* policy, float* value, hipStream_t s) {
  switch (n.filters) {
    case 64: return launch_f<MK, 64>(tiling, n, planes, legal, B, policy, value, s);
    case 128: return launch_f<MK, 128>(tiling, n, planes, legal, B, policy, value, s);
    case 256: return launch_f<MK, 256>(tiling, n, planes, legal, B, policy, value, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

bool az_mfma_supported(int dtype, int filters) {
  return (dtype >= 1 && dtype <= 3) && (filters == 64 || filters == 128 || filters == 256);
}

int az_mfma_boards_per_wg(int filters, int tiling) {
  if (tiling == 2) return 1;
  return filters == 256 ? 2 : 4;
}

hipError_t az_launch_mfma(int dtype, int tiling, const AzDevNet& n, const float* planes,
                          const uint8_t* legal, int B, float* policy, float* value,
                          hipStream_t s) {
  (void)hipGetLastError();
  switch (dtype) {
    case 1: return launch_mk<MK_BF16>(tiling, n, planes, legal, B, policy, value, s);
    case 2: return launch_mk<MK_I8>(tiling, n, planes, legal, B, policy, value, s);
    case 3: return launch_mk<MK_F8>(tiling, n, planes, legal, B, policy, value, s);
    default: return hipErrorInvalidValue;
  }
}
