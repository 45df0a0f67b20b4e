// Fused evaluation of the paper's deployed network on CDNA4 matrix cores
// (gfx950): 160-channel residual tower with global-pooling blocks, from-to
// policy head and WDL value head (Section 3.5 "Chess representation and
// outputs", Section 4.3 "Convolution, attention, and global context", "Three
// policy representations", "Value and training-only heads", Appendix D).
//
// One workgroup evaluates one board end to end, in one of two tilings.
// az_dep_kernel (large batches): one wave per workgroup, four such workgroups
// per compute unit for int8 (one per SIMD); the wave owns every output channel
// (five 32-channel MFMA blocks) and both half-board square blocks of every
// layer, so global pooling, the heads and both softmaxes need no exchange with
// other waves.  az_dep_kernel4 (small batches, where the batch offers about a
// board per compute unit): four waves, one per SIMD, share a layer's ten 32x32
// tiles, three at most per SIMD, and meet at a barrier per layer; they share
// the heads as well, exchanging operand fragments through LDS.
//
// Tower.  Every 3x3 convolution is an implicit GEMM D[ch][sq] = sum_k
// W[ch][k] X[k][sq], k = tap * C + c, with weights as the A operand (streamed
// from L2 in pre-packed fragment order through a ring of prefetched K steps)
// and the board's activations as the B operand, read from LDS rows [square][F
// channels].  Rows of 160 (int8) or 320 (bf16) bytes are not a power of two,
// so a row's 16-byte chunks are rotated by a few positions that depend on the
// square: the 16 lanes of a ds_read_b128 group (16 consecutive squares) then
// hit 16 different bank groups.  Out-of-board taps read a zero region at the
// bank slot their virtual square would use.
//
// Global pooling (every pool_every-th block).  After the first convolution's
// K loop, the pooled channels (the last F/4) are transposed through LDS (int8:
// the exact accumulators; bf16: their activations); one lane per pooled
// channel activates (int8, in float64) and reduces its row to a board sum
// (fp64) and maximum, and the projection c = Wg [mean, max] runs in fp64, one
// or two outputs per lane.  c is added to the regular channels' bias in the
// layer's constant slot (int8: in code units, in float64), so the epilogue
// that writes them takes it with the bias.
//
// bf16 networks carry the residual stream h as hi + lo: hi = bf16(h) is the
// convolution operand in LDS, lo = bf16(h - hi) stays in the registers of the
// lane that produces it (a 16-bit significand for the running sum).
//
// Heads.  The final tensor h (int8 codes, or the bf16 hi + lo parts) feeds one
// bf16 GEMM whose rows are the 128 token rows and
// the value rows.  The token, query and key products then run from registers:
// each accumulator tile is split into bf16 hi + lo parts and used directly as
// an MFMA operand, with the next weight matrix packed in the order the
// accumulator registers hold their rows (a permutation of the K dimension
// applied to both operands of the product); with four waves per board the
// tiles that cross waves go through LDS as those same fragments.  Query-key
// logits are written to LDS once, gathered through the action table, and
// soft-maxed over the legal actions in fp32; the WDL head runs on the vector
// ALUs.
#pragma once

#include "az_internal.h"
#include "az_mfma_common.h"

#include <math.h>

namespace {

constexpr int DF = 160;                         // filters
constexpr int DNMB = DF / 32;                   // 32-channel blocks
constexpr int DG = DF / 4;                      // pooled channels
constexpr int DFR = DF - DG;                    // regular channels of a pooling block
constexpr int DCP = AZ_DEP_MAX_IN_PLANES;       // stem input channels (padded)
constexpr int DD = AZ_DEP_TOKEN;                // token width
constexpr int DEMB = AZ_DEP_EMB_ROWS / 32;      // embedding row blocks (tokens + value rows)
constexpr int DTB = DD / 32;                    // token row blocks

typedef __attribute__((ext_vector_type(4))) float f32x4;

// Chunk position of logical 16-byte chunk lc in a row of RB bytes at swizzle
// sw: XOR for rows of 128 bytes, rotation modulo the row's chunk count for the
// 160- and 320-byte rows.
template <int RB>
struct Rot {
  static constexpr int NC = RB / 16;
  static constexpr int GC = gcd_c(NC, 16);      // NC*s mod 16 repeats every 16/GC squares
  static constexpr int SH = GC == 2 ? 3 : GC == 4 ? 2 : 1;
  static constexpr int RM = GC - 1;
  static_assert(RB == 160 || RB == 320, "rotated rows");
  static __device__ __forceinline__ int sw(int sq) { return (sq >> SH) & RM; }
  static __device__ __forceinline__ int pos(int lc, int sw) {
    const int x = lc + sw;
    return x >= NC ? x - NC : x;
  }
};

// swizzle of a 128-byte row (the stem's 64 bf16 input channels)
__device__ __forceinline__ int swz128(int sq) { return (sq >> 1) & 7; }

// LDS writes before, reads after, across every wave of the workgroup
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
}
// the same ordering within one wave (LDS writes by its lanes, reads by others)
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Board maximum (x) and sum (y) of pooled row pc of a pooling layer (first conv
// n_conv), read from LDS rows [pooled channel][square] with 16-byte chunks
// XOR-swizzled by the row.  int8 rows hold the exact accumulators, activated
// here in float64: act(acc * a[n] * s_w[f] + b1[f]); bf16 rows hold the
// activations.
template <bool QUANT>
__device__ __forceinline__ double2 pool_row(const AzDevNet& p, const float* pt, int pc, int n_conv) {
  double sum = 0.0, mx = 0.0;  // activations are >= 0
  // values made opaque to the compiler so that they are formed here, in the
  // pooling layer, not hoisted out of the block loop and held across the tower
  asm volatile("" : "+v"(pc));
  if constexpr (QUANT) {
    const size_t o = (size_t)n_conv * DF + DFR + pc;
    double cap = p.act_cap;
    asm volatile("" : "+v"(cap));
    const double pm = p.pool_m[o], pb = p.pool_b[o];
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int4 v = *reinterpret_cast<const int4*>(pt + pc * 64 + ((j ^ (pc & 15)) << 2));
      const int vv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const double a = clamp_d(__builtin_fma((double)vv[r], pm, pb), cap);
        sum += a;
        mx = __builtin_fmax(mx, a);
      }
    }
  } else {
    float mxf = 0.0f;
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const float4 v = *reinterpret_cast<const float4*>(pt + pc * 64 + ((j ^ (pc & 15)) << 2));
      sum += (double)v.x;
      sum += (double)v.y;
      sum += (double)v.z;
      sum += (double)v.w;
      mxf = fmaxf(mxf, fmaxf(fmaxf(v.x, v.y), fmaxf(v.z, v.w)));
    }
    mx = mxf;
  }
  return make_double2(mx, sum);
}

// Folds the projected context c[o] of a pooling layer into regular channel o's
// bias in the layer's constant slot: int8 slots hold qbias = b / a[n+1] in
// float64, so c enters in code units (c / a[n+1]); bf16 slots hold b in fp32.
template <bool QUANT>
__device__ __forceinline__ void add_context(const AzDevNet& p, float* kslot, int o, double c, int n_conv) {
  if constexpr (QUANT) reinterpret_cast<double*>(kslot)[o] += c * p.pool_cinv[n_conv];
  else kslot[o] += (float)c;
}

// bf16 hi and lo parts of eight fp32 values: x = hi + lo within 2^-16 |x|.
__device__ __forceinline__ void split8(const float (&x)[8], bf16x8& hi, bf16x8& lo) {
  uint32_t h[4], l[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const float a = x[2 * i], b = x[2 * i + 1];
    h[i] = pack_bf16x2(a, b);
    l[i] = pack_bf16x2(a - bf16_round(a), b - bf16_round(b));
  }
  hi = __builtin_bit_cast(bf16x8, make_uint4(h[0], h[1], h[2], h[3]));
  lo = __builtin_bit_cast(bf16x8, make_uint4(l[0], l[1], l[2], l[3]));
}

__device__ __forceinline__ f32x16 mma_bf16(const bf16x8& a, const bf16x8& b, const f32x16& c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ double shfl_xor_d(double v, int m) {
  const uint64_t u = __builtin_bit_cast(uint64_t, v);
  const uint32_t lo = (uint32_t)__shfl_xor((int)(uint32_t)u, m), hi = (uint32_t)__shfl_xor((int)(uint32_t)(u >> 32), m);
  return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}

template <int MK>
struct DepCfg {
  using T = Mk<MK>;
  static constexpr bool QUANT = MK != MK_BF16;
  static constexpr int RB = DF * T::ES;               // tower row bytes
  static constexpr int RBX = 2 * DF;                  // bf16 row bytes of the heads' input
  static constexpr int BUF = 64 * RB;
  static constexpr int OFF_H = 0, OFF_T = BUF, OFF_Z = 2 * BUF;
  static constexpr int ZB = (RB + 256 + 255) / 256 * 256;
  // per-layer epilogue constants: [bias F] floats, or for int8 [qbias F | qmul F
  // | qres, qhi] doubles (the float64 requantisation; the layer's two scalars
  // ride along so that the epilogue reads them from LDS: a load from global
  // memory there would wait behind the weight stream)
  static constexpr int KSLOT = QUANT ? 16 * DF + 16 : 4 * DF;
  static constexpr int OFF_K = OFF_Z + ZB;
  static constexpr int OFF_PG = OFF_K + 2 * KSLOT;    // pooled statistics, 2g doubles
  static constexpr int TOWER_END = OFF_PG + 2 * DG * 8;
  static constexpr int OFF_X = BUF;                   // heads' bf16 input: the lo part (bf16 networks)
  static constexpr int X_END = QUANT ? 0 : OFF_X + 64 * RBX;
  static constexpr int OFF_S = 0;                     // query-key logits [64][64] f32
  static constexpr int OFF_U = 64 * 64 * 4;           // value features [V][64] f32
  static constexpr int OFF_O = OFF_U + 32 * 64 * 4;   // promotion offsets [8][4] f32
  static constexpr int HEAD_END = OFF_O + 32 * 4;
  static constexpr int OFF_HC = (cmax(cmax(TOWER_END, X_END), HEAD_END) + 15) & ~15;  // head constants
  static constexpr int SMEM = OFF_HC + (2 * AZ_DEP_EMB_ROWS + 2 * DD) * 4;
  // four-wave tiling: operand fragments shared by the heads' waves (four planes of
  // 16 KB), past the one-wave layout
  static constexpr int OFF_Q4 = (SMEM + 255) & ~255;
  static constexpr int SMEM4 = OFF_Q4 + 4 * 16384;
  static_assert(OFF_T >= 64 * 128, "stem input fits in the T buffer");
  static constexpr int CPT = DF / T::KS;              // K steps per tap
  static constexpr int S = 9 * CPT;                   // K steps per layer
  static constexpr int NBUF = 3;                      // one-wave weight ring (steps), loaded NBUF-1 ahead
  static_assert((2 * S) % NBUF == 0, "every block's first conv starts at ring slot 0");
  static constexpr int STEP_BYTES = DNMB * 64 * T::FB;
  static constexpr size_t LAYER_BYTES = (size_t)S * STEP_BYTES;
};

// WDL value head of one board, one wave (lane = 0..63), from the value
// features U[c][sq] in LDS: y = relu(W1 u + b1), z = W2 y + b2, softmax over
// (win, draw, loss), value = W - L.
__device__ __forceinline__ void dep_wdl(const AzDevNet& p, const float* U, float* __restrict__ value,
                                        float* __restrict__ wdl, int b, int lane) {
  {
    const int H = p.value_hidden, NU = p.value_channels * 64;
    float z0 = 0.0f, z1 = 0.0f, z2 = 0.0f;
    for (int k0 = 0; k0 < H; k0 += 64) {
      const int k = k0 + lane;
      const bool ok = k < H;
      const int kk = ok ? k : 0;
      float y = p.wdl_fc1_b[kk];
      // fc1 row of unit kk in chunks of 16 inputs, the next chunk in flight
      // (NU is a multiple of 64)
      float wa[16], wb[16];
      auto ld = [&](float(&d)[16], int i0) {
#pragma unroll
        for (int t = 0; t < 16; ++t) d[t] = p.wdl_fc1_t[(size_t)(i0 + t) * H + kk];
      };
      ld(wa, 0);
      for (int i0 = 0; i0 < NU; i0 += 32) {
        ld(wb, i0 + 16);
#pragma unroll
        for (int t = 0; t < 16; ++t) y = __builtin_fmaf(wa[t], U[i0 + t], y);
        if (i0 + 32 < NU) ld(wa, i0 + 32);
#pragma unroll
        for (int t = 0; t < 16; ++t) y = __builtin_fmaf(wb[t], U[i0 + 16 + t], y);
      }
      y = ok ? fmaxf(y, 0.0f) : 0.0f;
      z0 = __builtin_fmaf(p.wdl_fc2_w[kk], y, z0);
      z1 = __builtin_fmaf(p.wdl_fc2_w[H + kk], y, z1);
      z2 = __builtin_fmaf(p.wdl_fc2_w[2 * H + kk], y, z2);
    }
    z0 = wave_sum(z0) + p.wdl_fc2_b[0];
    z1 = wave_sum(z1) + p.wdl_fc2_b[1];
    z2 = wave_sum(z2) + p.wdl_fc2_b[2];
    const float m = fmaxf(z0, fmaxf(z1, z2));
    const float e0 = expf(z0 - m), e1 = expf(z1 - m), e2 = expf(z2 - m);
    const float is = 1.0f / (e0 + e1 + e2);
    if (lane == 0) {
      const float pw = e0 * is, pd = e1 * is, pl = e2 * is;
      value[b] = pw - pl;
      if (wdl) {
        wdl[3 * (size_t)b + 0] = pw;
        wdl[3 * (size_t)b + 1] = pd;
        wdl[3 * (size_t)b + 2] = pl;
      }
    }
  }
}

// Heads of one board, run by one wave (lane = 0..63) once the final tower
// output h is in LDS (int8: codes in H; bf16: hi parts in H, lo parts in X):
// embedding, tokens, query-key logits and promotion offsets, legal-action
// softmax, WDL value head.
template <int MK>
__device__ __forceinline__ void dep_heads(const AzDevNet& p, uint8_t* smem, const uint8_t* __restrict__ legal,
                                          float* __restrict__ policy, float* __restrict__ value,
                                          float* __restrict__ wdl, int b, int lane_in) {
  using C = DepCfg<MK>;
  using R = Rot<C::RB>;
  using RX = Rot<C::RBX>;
  constexpr bool QUANT = C::QUANT;
  constexpr int RB = C::RB, OFF_H = C::OFF_H;
  // the lane index, opaque to the compiler here, so that the heads' lane-dependent
  // addresses are computed in the heads instead of being shared with the stem's
  // and held (or spilled) across the tower
  int lane = lane_in;
  asm volatile("" : "+v"(lane));
  const int l32 = lane & 31, lhi = lane >> 5;

  // ---- embedding: E[row][sq] = sum_f Wemb[row][f] h[f][sq], rows = tokens then value channels
  f32x16 tok[DTB][2];   // token rows (accumulators, then values)
  f32x16 uacc[2];       // value rows 128..159
  {
    const uint8_t* ew = static_cast<const uint8_t*>(p.emb_w) + (size_t)lane * 16;
    // A fragments of K step s in ring slot s % 4, loaded three steps ahead
    constexpr int ES = DF / 16, ER = 4;
    bf16x8 awr[ER][DEMB];
    auto load_e = [&](int st) {
#pragma unroll
      for (int m = 0; m < DEMB; ++m) awr[st % ER][m] = g_frag<MK_BF16>(ew + (st * DEMB + m) * 64 * 16);
    };
#pragma unroll
    for (int st = 0; st < ER - 1; ++st) load_e(st);
#pragma unroll
    for (int s = 0; s < ES; ++s) {
      if (s + ER - 1 < ES) load_e(s + ER - 1);
      const bf16x8(&aw)[DEMB] = awr[s % ER];
      bf16x8 bx[2], bh[2];
#pragma unroll
      for (int n = 0; n < 2; ++n) {
        const int j = n * 32 + l32;
        if constexpr (QUANT) {
          // eight codes of channels 16 s + 8 lhi .. + 7, exact in bf16
          const uint2 v = *reinterpret_cast<const uint2*>(smem + OFF_H + j * RB + (R::pos(s, R::sw(j)) << 4) + 8 * lhi);
          bx[n] = __builtin_bit_cast(
              bf16x8, make_uint4(pack_bf16x2(code_value<MK, 0>(v.x), code_value<MK, 1>(v.x)),
                                 pack_bf16x2(code_value<MK, 2>(v.x), code_value<MK, 3>(v.x)),
                                 pack_bf16x2(code_value<MK, 0>(v.y), code_value<MK, 1>(v.y)),
                                 pack_bf16x2(code_value<MK, 2>(v.y), code_value<MK, 3>(v.y))));
        } else {
          bx[n] = *reinterpret_cast<const bf16x8*>(smem + C::OFF_X + j * C::RBX + (RX::pos(2 * s + lhi, RX::sw(j)) << 4));
          bh[n] = *reinterpret_cast<const bf16x8*>(smem + OFF_H + j * C::RBX + (RX::pos(2 * s + lhi, RX::sw(j)) << 4));
        }
      }
#pragma unroll
      for (int n = 0; n < 2; ++n) {
#pragma unroll
        for (int m = 0; m < DTB; ++m) {
          tok[m][n] = mma_bf16(aw[m], bx[n], s == 0 ? f32x16{} : tok[m][n]);
          if constexpr (!QUANT) tok[m][n] = mma_bf16(aw[m], bh[n], tok[m][n]);
        }
        uacc[n] = mma_bf16(aw[DTB], bx[n], s == 0 ? f32x16{} : uacc[n]);
        if constexpr (!QUANT) uacc[n] = mma_bf16(aw[DTB], bh[n], uacc[n]);
      }
    }
  }
  wave_sync();  // H and X are dead from here on

  // token values relu(acc * scale + bias); value features u[c][sq] to LDS
  const float* HC = reinterpret_cast<const float*>(smem + C::OFF_HC);
  {
#pragma unroll
    for (int m = 0; m < DTB; ++m)
#pragma unroll
      for (int jq = 0; jq < 4; ++jq) {
        const int r0 = 32 * m + 8 * jq + 4 * lhi;
        const float4 sc = *reinterpret_cast<const float4*>(HC + r0);
        const float4 bc = *reinterpret_cast<const float4*>(HC + AZ_DEP_EMB_ROWS + r0);
        const float sv[4] = {sc.x, sc.y, sc.z, sc.w}, bv[4] = {bc.x, bc.y, bc.z, bc.w};
#pragma unroll
        for (int n = 0; n < 2; ++n)
#pragma unroll
          for (int r = 0; r < 4; ++r) tok[m][n][4 * jq + r] = fmaxf(__builtin_fmaf(tok[m][n][4 * jq + r], sv[r], bv[r]), 0.0f);
      }
    float* U = reinterpret_cast<float*>(smem + C::OFF_U);
    const int V = p.value_channels;
#pragma unroll
    for (int jq = 0; jq < 4; ++jq) {
      const int r0 = DD + 8 * jq + 4 * lhi;
      const float4 sc = *reinterpret_cast<const float4*>(HC + r0);
      const float4 bc = *reinterpret_cast<const float4*>(HC + AZ_DEP_EMB_ROWS + r0);
      const float sv[4] = {sc.x, sc.y, sc.z, sc.w}, bv[4] = {bc.x, bc.y, bc.z, bc.w};
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int ch = 8 * jq + 4 * lhi + r;
        if (ch < V) {
#pragma unroll
          for (int n = 0; n < 2; ++n) {
            float u = __builtin_fmaf(uacc[n][4 * jq + r], sv[r], bv[r]);
            if (p.value_conv_relu) u = fmaxf(u, 0.0f);
            U[ch * 64 + n * 32 + l32] = u;
          }
        }
      }
    }
  }

  // The token values as split bf16 operand fragments: K step s (0..7) of the
  // products below holds positions 8s .. 8s+7 of the lane's 64 token values
  // (the accumulators' register order), as x = hi + lo.
  bf16x8 tkh[DD / 16][2], tkl[DD / 16][2];
#pragma unroll
  for (int st = 0; st < DD / 16; ++st)
#pragma unroll
    for (int n = 0; n < 2; ++n) {
      float x[8];
#pragma unroll
      for (int t = 0; t < 8; ++t) x[t] = tok[(8 * st + t) / 16][n][(8 * st + t) % 16];
      split8(x, tkh[st][n], tkl[st][n]);
    }

  // action table entries and legal-mask words of the softmax, in flight during
  // the last query / key block's products
  constexpr int NA = AZ_FROMTO_ACTIONS, NIT = (NA + 255) / 256;
  uint4 tbl[NIT];
  uint32_t mkw[NIT];
  auto load_actions = [&]() {
    const uint8_t* lg = legal + (size_t)b * NA;
#pragma unroll
    for (int i = 0; i < NIT; ++i) {
      const int a0 = 256 * i + 4 * lane;
      const bool in = a0 < NA;
      tbl[i] = *reinterpret_cast<const uint4*>(p.actions + (in ? a0 : 0));
      const uint32_t mk0 = *reinterpret_cast<const uint32_t*>(lg + (in ? a0 : 0));  // clamped, unconditional
      mkw[i] = in ? mk0 : 0u;
    }
  };

  // Per 32-row block m of Q^T = Wq tok^T + bq and K^T = Wk tok^T + bk (rows in
  // the token accumulators' register order), then the two K steps 2m, 2m+1 of
  //   S[f][t] = sum_d Q[f][d] K[t][d]      (hi*hi + hi*lo + lo*hi)
  //   O^T[k][t] = sum_d Wp[k][d] K[t][d]   (promotion offsets, last row's destinations)
  // that block holds.  Every accumulator runs the same chain of products as
  // when all blocks are computed at once (the four-wave heads do that), with
  // only one block of Q and K live at a time.
  f32x16 Sa[2][2], Oa;
  {
    const uint8_t* qp = static_cast<const uint8_t*>(p.q_w) + (size_t)lane * 16;
    const uint8_t* kp = static_cast<const uint8_t*>(p.k_w) + (size_t)lane * 16;
    const uint8_t* pw = static_cast<const uint8_t*>(p.p_w) + (size_t)lane * 16;
    constexpr int QS = DD / 16, QR = 2;
#pragma unroll
    for (int m = 0; m < DTB; ++m) {
      if (m == DTB - 1) load_actions();
      const bf16x8 apw0 = g_frag<MK_BF16>(pw + (2 * m) * 64 * 16), apw1 = g_frag<MK_BF16>(pw + (2 * m + 1) * 64 * 16);
      f32x16 Qm[2], Km[2];
      // A fragments of K step s in ring slot s % 2, loaded one step ahead
      bf16x8 aqr[QR], akr[QR];
      auto load_qk = [&](int st) {
        aqr[st % QR] = g_frag<MK_BF16>(qp + (st * DTB + m) * 64 * 16);
        akr[st % QR] = g_frag<MK_BF16>(kp + (st * DTB + m) * 64 * 16);
      };
      load_qk(0);
#pragma unroll
      for (int st = 0; st < QS; ++st) {
        if (st + 1 < QS) load_qk(st + 1);
#pragma unroll
        for (int n = 0; n < 2; ++n) {
          Qm[n] = mma_bf16(aqr[st % QR], tkh[st][n], st == 0 ? f32x16{} : Qm[n]);
          Qm[n] = mma_bf16(aqr[st % QR], tkl[st][n], Qm[n]);
          Km[n] = mma_bf16(akr[st % QR], tkh[st][n], st == 0 ? f32x16{} : Km[n]);
          Km[n] = mma_bf16(akr[st % QR], tkl[st][n], Km[n]);
        }
      }
#pragma unroll
      for (int jq = 0; jq < 4; ++jq) {
        const int r0 = 32 * m + 8 * jq + 4 * lhi;
        const float4 bq = *reinterpret_cast<const float4*>(HC + 2 * AZ_DEP_EMB_ROWS + r0);
        const float4 bk = *reinterpret_cast<const float4*>(HC + 2 * AZ_DEP_EMB_ROWS + DD + r0);
        const float qv[4] = {bq.x, bq.y, bq.z, bq.w}, kv[4] = {bk.x, bk.y, bk.z, bk.w};
#pragma unroll
        for (int n = 0; n < 2; ++n)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            Qm[n][4 * jq + r] += qv[r];
            Km[n][4 * jq + r] += kv[r];
          }
      }
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int s = 2 * m + h;
        bf16x8 qh[2], ql[2], kh[2], kl[2];
#pragma unroll
        for (int n = 0; n < 2; ++n) {
          float xq[8], xk[8];
#pragma unroll
          for (int t = 0; t < 8; ++t) {
            xq[t] = Qm[n][8 * h + t];
            xk[t] = Km[n][8 * h + t];
          }
          split8(xq, qh[n], ql[n]);
          split8(xk, kh[n], kl[n]);
        }
#pragma unroll
        for (int mf = 0; mf < 2; ++mf)
#pragma unroll
          for (int nt = 0; nt < 2; ++nt) {
            Sa[mf][nt] = mma_bf16(qh[mf], kh[nt], s == 0 ? f32x16{} : Sa[mf][nt]);
            Sa[mf][nt] = mma_bf16(qh[mf], kl[nt], Sa[mf][nt]);
            Sa[mf][nt] = mma_bf16(ql[mf], kh[nt], Sa[mf][nt]);
          }
        Oa = mma_bf16(h ? apw1 : apw0, kh[1], s == 0 ? f32x16{} : Oa);
        Oa = mma_bf16(h ? apw1 : apw0, kl[1], Oa);
      }
    }
  }
  // logits pre-scaled by log2(e) for the exp2 softmax
  {
    const float log2e = 1.4426950408889634f;
    const float ss = log2e / sqrtf((float)DD);
    float* S = reinterpret_cast<float*>(smem + C::OFF_S);
#pragma unroll
    for (int mf = 0; mf < 2; ++mf)
#pragma unroll
      for (int nt = 0; nt < 2; ++nt)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int f = 32 * mf + 8 * (v / 4) + 4 * lhi + v % 4, t = 32 * nt + l32;
          S[f * 64 + t] = Sa[mf][nt][v] * ss;
        }
    float* O = reinterpret_cast<float*>(smem + C::OFF_O);
    if (lhi == 0 && l32 >= 24) {
#pragma unroll
      for (int k = 0; k < 4; ++k) O[(l32 - 24) * 4 + k] = Oa[k] * log2e;
    }
  }
  wave_sync();

  // ---- legal-action softmax: lane owns the runs of 4 actions at 256 i + 4 lane
  {
    const float* S = reinterpret_cast<const float*>(smem + C::OFF_S);
    const float* O = reinterpret_cast<const float*>(smem + C::OFF_O);
    float e[NIT][4];
    float mx = -INFINITY;
#pragma unroll
    for (int i = 0; i < NIT; ++i) {
      const int a0 = 256 * i + 4 * lane;
      const bool in = a0 < NA;  // NA is a multiple of 4
      const uint4 tb = tbl[i];
      const uint32_t mk = mkw[i];
      const uint32_t te[4] = {tb.x, tb.y, tb.z, tb.w};
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const uint32_t x = te[r], pr = x >> 12;
        const float z = S[x & 4095u] + (pr ? O[pr - 1] : 0.0f);
        const bool ok = in && ((mk >> (8 * r)) & 0xffu);
        e[i][r] = ok ? z : -INFINITY;
        mx = fmaxf(mx, e[i][r]);
      }
    }
    mx = wave_max(mx);
    const float msub = mx == -INFINITY ? 0.0f : mx;
    float sum = 0.0f;
#pragma unroll
    for (int i = 0; i < NIT; ++i)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        e[i][r] = __builtin_amdgcn_exp2f(e[i][r] - msub);  // exp2(-inf) = 0
        sum += e[i][r];
      }
    sum = wave_sum(sum);
    const float inv = sum > 0.0f ? 1.0f / sum : 0.0f;
    float* pol = policy + (size_t)b * NA;
#pragma unroll
    for (int i = 0; i < NIT; ++i) {
      const int a0 = 256 * i + 4 * lane;
      if (a0 < NA)
        *reinterpret_cast<float4*>(pol + a0) = make_float4(e[i][0] * inv, e[i][1] * inv, e[i][2] * inv, e[i][3] * inv);
    }
  }

  // ---- WDL head
  dep_wdl(p, reinterpret_cast<const float*>(smem + C::OFF_U), value, wdl, b, lane);
}

// Heads of one board shared by the four waves of az_dep_kernel4 (wave = 0..3,
// lane = 0..63), once the final tower output h is in LDS.  The arithmetic is
// dep_heads' operation for operation: every accumulator tile runs the same
// chain of products, split operands are split the same way, and the softmax
// normaliser is summed in the same order, so the outputs are bitwise the same.
// The work is spread as the tower's is: wave w owns token / query / key block w
// and one 32x32 tile of the logits S; operands that cross waves go through LDS
// as the very fragments a single wave would have taken from its registers
// (fragment set [square block][K step][lane] of 16 bytes).
template <int MK>
__device__ __forceinline__ void dep_heads4(const AzDevNet& p, uint8_t* smem, const uint8_t* __restrict__ legal,
                                           float* __restrict__ policy, float* __restrict__ value,
                                           float* __restrict__ wdl, int b, int wave, int lane) {
  using C = DepCfg<MK>;
  using R = Rot<C::RB>;
  using RX = Rot<C::RBX>;
  constexpr bool QUANT = C::QUANT;
  constexpr int RB = C::RB, OFF_H = C::OFF_H;
  constexpr int FS = 64 * 16;                   // bytes of one fragment set
  static_assert(DTB == 4, "one token block per wave");
  const int l32 = lane & 31, lhi = lane >> 5;
  const float* HC = reinterpret_cast<const float*>(smem + C::OFF_HC);
  uint8_t* const q4 = smem + C::OFF_Q4;
  // fragment set of K step s (0..7) of square block n in one of the four 16 KB planes
  auto fset = [&](int plane, int n, int s) { return q4 + plane * 16384 + ((n * 8 + s) * 64 + lane) * 16; };

  // action table entries and legal-mask words of this wave's two groups of 256
  // actions (actions 256 i + 4 lane .. + 3), in flight during the products
  constexpr int NA = AZ_FROMTO_ACTIONS, NIT = (NA + 255) / 256, GW = NIT / 4;
  static_assert(NIT % 4 == 0, "action groups per wave");
  uint4 tbl[GW];
  uint32_t mkw[GW];
  {
    const uint8_t* lg = legal + (size_t)b * NA;
#pragma unroll
    for (int g = 0; g < GW; ++g) {
      const int a0 = 256 * (wave * GW + g) + 4 * lane;
      const bool in = a0 < NA;
      tbl[g] = *reinterpret_cast<const uint4*>(p.actions + (in ? a0 : 0));
      const uint32_t mk0 = *reinterpret_cast<const uint32_t*>(lg + (in ? a0 : 0));  // clamped, unconditional
      mkw[g] = in ? mk0 : 0u;
    }
  }

  // every weight fragment of the wave's embedding rows and query / key rows,
  // issued at once: the heads then wait for one load latency, not one per step
  constexpr int ES = DF / 16, QS = DD / 16;
  bf16x8 awe[ES][2], aq[QS], ak[QS];
  {
    const uint8_t* ew = static_cast<const uint8_t*>(p.emb_w) + (size_t)lane * 16;
    const uint8_t* qp = static_cast<const uint8_t*>(p.q_w) + (size_t)lane * 16;
    const uint8_t* kp = static_cast<const uint8_t*>(p.k_w) + (size_t)lane * 16;
#pragma unroll
    for (int st = 0; st < ES; ++st) {
      awe[st][0] = g_frag<MK_BF16>(ew + (st * DEMB + wave) * FS);
      awe[st][1] = g_frag<MK_BF16>(ew + (st * DEMB + DTB) * FS);
    }
#pragma unroll
    for (int st = 0; st < QS; ++st) {
      aq[st] = g_frag<MK_BF16>(qp + (st * DTB + wave) * FS);
      ak[st] = g_frag<MK_BF16>(kp + (st * DTB + wave) * FS);
    }
  }

  // ---- embedding: token rows of block wave (both square blocks) and the value
  // rows on square block wave & 1 (kept by waves 0 and 1)
  const int nv = wave & 1;
  f32x16 tk[2], ua;
  {
#pragma unroll
    for (int s = 0; s < ES; ++s) {
      const bf16x8(&aw)[2] = awe[s];
      bf16x8 bx[2], bh[2];
#pragma unroll
      for (int n = 0; n < 2; ++n) {
        const int j = n * 32 + l32;
        if constexpr (QUANT) {
          const uint2 v = *reinterpret_cast<const uint2*>(smem + OFF_H + j * RB + (R::pos(s, R::sw(j)) << 4) + 8 * lhi);
          bx[n] = __builtin_bit_cast(
              bf16x8, make_uint4(pack_bf16x2(code_value<MK, 0>(v.x), code_value<MK, 1>(v.x)),
                                 pack_bf16x2(code_value<MK, 2>(v.x), code_value<MK, 3>(v.x)),
                                 pack_bf16x2(code_value<MK, 0>(v.y), code_value<MK, 1>(v.y)),
                                 pack_bf16x2(code_value<MK, 2>(v.y), code_value<MK, 3>(v.y))));
        } else {
          bx[n] = *reinterpret_cast<const bf16x8*>(smem + C::OFF_X + j * C::RBX + (RX::pos(2 * s + lhi, RX::sw(j)) << 4));
          bh[n] = *reinterpret_cast<const bf16x8*>(smem + OFF_H + j * C::RBX + (RX::pos(2 * s + lhi, RX::sw(j)) << 4));
        }
      }
#pragma unroll
      for (int n = 0; n < 2; ++n) {
        tk[n] = mma_bf16(aw[0], bx[n], s == 0 ? f32x16{} : tk[n]);
        if constexpr (!QUANT) tk[n] = mma_bf16(aw[0], bh[n], tk[n]);
      }
      const bf16x8 bxv = nv ? bx[1] : bx[0];
      ua = mma_bf16(aw[1], bxv, s == 0 ? f32x16{} : ua);
      if constexpr (!QUANT) {
        const bf16x8 bhv = nv ? bh[1] : bh[0];
        ua = mma_bf16(aw[1], bhv, ua);
      }
    }
  }
  wave_lds_sync();  // H and X are dead from here on

  // token values relu(acc * scale + bias), as the query / key products' B
  // fragments of K steps 2 wave and 2 wave + 1; value features u[c][sq] to LDS
  {
#pragma unroll
    for (int jq = 0; jq < 4; ++jq) {
      const int r0 = 32 * wave + 8 * jq + 4 * lhi;
      const float4 sc = *reinterpret_cast<const float4*>(HC + r0);
      const float4 bc = *reinterpret_cast<const float4*>(HC + AZ_DEP_EMB_ROWS + r0);
      const float sv[4] = {sc.x, sc.y, sc.z, sc.w}, bv[4] = {bc.x, bc.y, bc.z, bc.w};
#pragma unroll
      for (int n = 0; n < 2; ++n)
#pragma unroll
        for (int r = 0; r < 4; ++r) tk[n][4 * jq + r] = fmaxf(__builtin_fmaf(tk[n][4 * jq + r], sv[r], bv[r]), 0.0f);
    }
#pragma unroll
    for (int n = 0; n < 2; ++n)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        float x[8];
#pragma unroll
        for (int t = 0; t < 8; ++t) x[t] = tk[n][8 * h + t];
        bf16x8 hi, lo;
        split8(x, hi, lo);
        *reinterpret_cast<bf16x8*>(fset(0, n, 2 * wave + h)) = hi;
        *reinterpret_cast<bf16x8*>(fset(1, n, 2 * wave + h)) = lo;
      }
    if (wave < 2) {
      float* U = reinterpret_cast<float*>(smem + C::OFF_U);
      const int V = p.value_channels;
#pragma unroll
      for (int jq = 0; jq < 4; ++jq) {
        const int r0 = DD + 8 * jq + 4 * lhi;
        const float4 sc = *reinterpret_cast<const float4*>(HC + r0);
        const float4 bc = *reinterpret_cast<const float4*>(HC + AZ_DEP_EMB_ROWS + r0);
        const float sv[4] = {sc.x, sc.y, sc.z, sc.w}, bv[4] = {bc.x, bc.y, bc.z, bc.w};
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int ch = 8 * jq + 4 * lhi + r;
          if (ch < V) {
            float u = __builtin_fmaf(ua[4 * jq + r], sv[r], bv[r]);
            if (p.value_conv_relu) u = fmaxf(u, 0.0f);
            U[ch * 64 + nv * 32 + l32] = u;
          }
        }
      }
    }
  }
  wave_lds_sync();

  // query and key block wave: Q^T = Wq tok^T + bq, K^T = Wk tok^T + bk over the
  // eight token K steps (hi, then lo)
  f32x16 Qa[2], Ka[2];
  {
#pragma unroll
    for (int s = 0; s < QS; ++s) {
#pragma unroll
      for (int n = 0; n < 2; ++n) {
        const bf16x8 xh = *reinterpret_cast<const bf16x8*>(fset(0, n, s));
        const bf16x8 xl = *reinterpret_cast<const bf16x8*>(fset(1, n, s));
        Qa[n] = mma_bf16(aq[s], xh, s == 0 ? f32x16{} : Qa[n]);
        Qa[n] = mma_bf16(aq[s], xl, Qa[n]);
        Ka[n] = mma_bf16(ak[s], xh, s == 0 ? f32x16{} : Ka[n]);
        Ka[n] = mma_bf16(ak[s], xl, Ka[n]);
      }
    }
#pragma unroll
    for (int jq = 0; jq < 4; ++jq) {
      const int r0 = 32 * wave + 8 * jq + 4 * lhi;
      const float4 bq = *reinterpret_cast<const float4*>(HC + 2 * AZ_DEP_EMB_ROWS + r0);
      const float4 bk = *reinterpret_cast<const float4*>(HC + 2 * AZ_DEP_EMB_ROWS + DD + r0);
      const float qv[4] = {bq.x, bq.y, bq.z, bq.w}, kv[4] = {bk.x, bk.y, bk.z, bk.w};
#pragma unroll
      for (int n = 0; n < 2; ++n)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          Qa[n][4 * jq + r] += qv[r];
          Ka[n][4 * jq + r] += kv[r];
        }
    }
  }
  wave_lds_sync();  // token fragments dead
  // the logits' A (query) and B (key) fragments of K steps 2 wave, 2 wave + 1
#pragma unroll
  for (int n = 0; n < 2; ++n)
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      float x[8], y[8];
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        x[t] = Qa[n][8 * h + t];
        y[t] = Ka[n][8 * h + t];
      }
      bf16x8 qh, ql, kh, kl;
      split8(x, qh, ql);
      split8(y, kh, kl);
      *reinterpret_cast<bf16x8*>(fset(0, n, 2 * wave + h)) = qh;
      *reinterpret_cast<bf16x8*>(fset(1, n, 2 * wave + h)) = ql;
      *reinterpret_cast<bf16x8*>(fset(2, n, 2 * wave + h)) = kh;
      *reinterpret_cast<bf16x8*>(fset(3, n, 2 * wave + h)) = kl;
    }
  wave_lds_sync();

  // S tile (mf, nt) = (wave >> 1, wave & 1): S[f][t] = sum_d Q[f][d] K[t][d]
  // (hi*hi + hi*lo + lo*hi); the promotion offsets O^T = Wp K^T of the last row's
  // destinations (square block 1, written by wave 3)
  {
    const int mf = wave >> 1, nt = wave & 1;
    const uint8_t* pw = static_cast<const uint8_t*>(p.p_w) + (size_t)lane * 16;
    bf16x8 apw[DD / 16];
#pragma unroll
    for (int s = 0; s < DD / 16; ++s) apw[s] = g_frag<MK_BF16>(pw + s * FS);
    f32x16 Sa, Oa;
#pragma unroll
    for (int s = 0; s < DD / 16; ++s) {
      const bf16x8 qh = *reinterpret_cast<const bf16x8*>(fset(0, mf, s));
      const bf16x8 ql = *reinterpret_cast<const bf16x8*>(fset(1, mf, s));
      const bf16x8 kh = *reinterpret_cast<const bf16x8*>(fset(2, nt, s));
      const bf16x8 kl = *reinterpret_cast<const bf16x8*>(fset(3, nt, s));
      Sa = mma_bf16(qh, kh, s == 0 ? f32x16{} : Sa);
      Sa = mma_bf16(qh, kl, Sa);
      Sa = mma_bf16(ql, kh, Sa);
      Oa = mma_bf16(apw[s], kh, s == 0 ? f32x16{} : Oa);
      Oa = mma_bf16(apw[s], kl, Oa);
    }
    // logits pre-scaled by log2(e) for the exp2 softmax
    const float log2e = 1.4426950408889634f;
    const float ss = log2e / sqrtf((float)DD);
    float* S = reinterpret_cast<float*>(smem + C::OFF_S);
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      const int f = 32 * mf + 8 * (v / 4) + 4 * lhi + v % 4, t = 32 * nt + l32;
      S[f * 64 + t] = Sa[v] * ss;
    }
    float* O = reinterpret_cast<float*>(smem + C::OFF_O);
    if (wave == 3 && lhi == 0 && l32 >= 24) {
#pragma unroll
      for (int k = 0; k < 4; ++k) O[(l32 - 24) * 4 + k] = Oa[k] * log2e;
    }
  }
  wave_lds_sync();  // query / key fragments dead

  // ---- legal-action softmax: wave w gathers and exponentiates groups 2w, 2w + 1;
  // the maximum is exact in any order, the normaliser is summed by wave 0 over all
  // groups in the one-wave order
  float* E = reinterpret_cast<float*>(q4);            // numerators, 2048 slots
  float* MX = reinterpret_cast<float*>(q4 + 8192);    // per-wave maxima, then 1 / sum
  {
    const float* S = reinterpret_cast<const float*>(smem + C::OFF_S);
    const float* O = reinterpret_cast<const float*>(smem + C::OFF_O);
    float e[GW][4];
    float mx = -INFINITY;
#pragma unroll
    for (int g = 0; g < GW; ++g) {
      const int a0 = 256 * (wave * GW + g) + 4 * lane;
      const bool in = a0 < NA;  // NA is a multiple of 4
      const uint4 tb = tbl[g];
      const uint32_t mk = mkw[g];
      const uint32_t te[4] = {tb.x, tb.y, tb.z, tb.w};
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const uint32_t x = te[r], pr = x >> 12;
        const float z = S[x & 4095u] + (pr ? O[pr - 1] : 0.0f);
        const bool ok = in && ((mk >> (8 * r)) & 0xffu);
        e[g][r] = ok ? z : -INFINITY;
        mx = fmaxf(mx, e[g][r]);
      }
    }
    mx = wave_max(mx);
    if (lane == 0) MX[wave] = mx;
    wave_lds_sync();
    mx = fmaxf(fmaxf(MX[0], MX[1]), fmaxf(MX[2], MX[3]));
    const float msub = mx == -INFINITY ? 0.0f : mx;
#pragma unroll
    for (int g = 0; g < GW; ++g) {
#pragma unroll
      for (int r = 0; r < 4; ++r) e[g][r] = __builtin_amdgcn_exp2f(e[g][r] - msub);  // exp2(-inf) = 0
      *reinterpret_cast<float4*>(E + 256 * (wave * GW + g) + 4 * lane) = make_float4(e[g][0], e[g][1], e[g][2], e[g][3]);
    }
    wave_lds_sync();
    if (wave == 0) {
      float sum = 0.0f;
#pragma unroll
      for (int i = 0; i < NIT; ++i) {
        const float4 v = *reinterpret_cast<const float4*>(E + 256 * i + 4 * lane);
        sum += v.x;
        sum += v.y;
        sum += v.z;
        sum += v.w;
      }
      sum = wave_sum(sum);
      if (lane == 0) MX[4] = sum > 0.0f ? 1.0f / sum : 0.0f;
    }
    wave_lds_sync();
    const float inv = MX[4];
    float* pol = policy + (size_t)b * NA;
#pragma unroll
    for (int g = 0; g < GW; ++g) {
      const int a0 = 256 * (wave * GW + g) + 4 * lane;
      if (a0 < NA)
        *reinterpret_cast<float4*>(pol + a0) = make_float4(e[g][0] * inv, e[g][1] * inv, e[g][2] * inv, e[g][3] * inv);
    }
  }

  // ---- WDL head (wave 1): y = relu(W1 u + b1), z = W2 y + b2, softmax, value = W - L
  if (wave == 1) dep_wdl(p, reinterpret_cast<const float*>(smem + C::OFF_U), value, wdl, b, lane);
}

template <int MK>
__global__ __attribute__((amdgpu_flat_work_group_size(64, 64), amdgpu_waves_per_eu(1, 1))) void
az_dep_kernel(AzDevNet p, const float* __restrict__ planes, const uint8_t* __restrict__ legal,
              float* __restrict__ policy, float* __restrict__ value, float* __restrict__ wdl) {
  using C = DepCfg<MK>;
  using T = typename C::T;
  using frag_t = typename T::frag;
  using acc_t = typename T::acc;
  using R = Rot<C::RB>;
  constexpr bool QUANT = C::QUANT;
  constexpr int RB = C::RB, OFF_H = C::OFF_H, OFF_T = C::OFF_T, OFF_Z = C::OFF_Z;

  __shared__ __attribute__((aligned(16))) uint8_t smem[C::SMEM];

  constexpr int NBW = 2;  // half-board square blocks (the wave owns the whole board)
  const int lane = threadIdx.x;
  const int l32 = lane & 31, lhi = lane >> 5;
  const int b = blockIdx.x;
  const int Cin = p.in_planes;
  const float cap = p.act_cap;

  // residual stream of the board (bf16 networks): h = hi + lo, hi = bf16(h) in
  // the H buffer (the convolution operand), lo = bf16(h - hi) packed here, two
  // per register: [block][half][run of 4 channels][2]
  uint32_t rlo[QUANT ? 1 : DNMB][QUANT ? 1 : NBW][QUANT ? 1 : 8];

  // ---- ingest: zero region, planes -> bf16 [square][64 channels] at OFF_T
  for (int i = lane; i < C::ZB / 16; i += 64)
    *reinterpret_cast<i32x4*>(smem + OFF_Z + i * 16) = i32x4{0, 0, 0, 0};
  {
    // item k = planes 8k..8k+7: lane = square, eight coalesced loads, one
    // 16-byte store
    constexpr int KI = DCP / 8;
    float pv[KI][8];
#pragma unroll
    for (int ki = 0; ki < KI; ++ki)
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const int c = 8 * ki + t;
        const bool ok = c < Cin;
        const float x = planes[((size_t)b * Cin + (ok ? c : 0)) * 64 + lane];
        pv[ki][t] = ok ? x : 0.0f;
      }
#pragma unroll
    for (int ki = 0; ki < KI; ++ki) {
      const int k = ki;
      *reinterpret_cast<uint4*>(smem + OFF_T + lane * 128 + ((k ^ swz128(lane)) << 4)) =
          make_uint4(pack_bf16x2(pv[ki][0], pv[ki][1]), pack_bf16x2(pv[ki][2], pv[ki][3]),
                     pack_bf16x2(pv[ki][4], pv[ki][5]), pack_bf16x2(pv[ki][6], pv[ki][7]));
    }
  }

  // tower weight ring: K step i of the stream lives in A[i % NBUF].  The stream
  // is read through a buffer resource: the lane's offset is a constant VGPR, the
  // step's byte offset a scalar and the block's a literal, so a step's five
  // loads cost no vector address arithmetic.
  constexpr int NBUF = C::NBUF;
  const __amdgpu_buffer_rsrc_t twr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<void*>(p.tower_w), (short)0, (int)(2 * p.blocks * C::LAYER_BYTES), 0x00020000);
  const int tvoff = lane * T::FB;
  frag_t A[NBUF][DNMB];
  auto load_step = [&](frag_t(&dst)[DNMB], int soff) {
#pragma unroll
    for (int m = 0; m < DNMB; ++m)
      dst[m] = __builtin_bit_cast(frag_t, __builtin_amdgcn_raw_buffer_load_b128(twr, tvoff, soff + m * 64 * T::FB, 0));
  };
  // per-layer epilogue constants of conv index k (0 = stem): [bias F] floats, or
  // [qbias F | qmul F] doubles, as lane-held 16-byte chunks loaded at the start
  // of a layer and parked in LDS before its barrier
  constexpr int KV = C::KSLOT / 16;                  // 16-byte chunks per slot
  constexpr int KPL = (KV + 63) / 64;                // per lane
  auto load_consts = [&](int k, float4(&dst)[KPL]) {
#pragma unroll
    for (int t = 0; t < KPL; ++t) {
      const int i = lane + 64 * t;
      const void* src;
      if constexpr (QUANT)
        src = i < DF / 2 ? p.qbias + (size_t)k * DF + 2 * i
              : i < DF   ? p.qmul + (size_t)k * DF + 2 * (i - DF / 2)
                         : p.qext + 2 * (size_t)k;
      else src = p.bias + (size_t)k * DF + 4 * i;
      dst[t] = i < KV ? *reinterpret_cast<const float4*>(src) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  };
  auto store_consts = [&](int slot, const float4(&v)[KPL]) {
    float4* dst = reinterpret_cast<float4*>(smem + C::OFF_K + slot * C::KSLOT);
#pragma unroll
    for (int t = 0; t < KPL; ++t)
      if (lane + 64 * t < KV) dst[lane + 64 * t] = v[t];
  };
  // head constants, staged once: embedding row scale and bias, query and key biases
  {
    float* hc = reinterpret_cast<float*>(smem + C::OFF_HC);
    for (int i = lane; i < AZ_DEP_EMB_ROWS; i += 64) {
      hc[i] = p.emb_sc[i];
      hc[AZ_DEP_EMB_ROWS + i] = p.emb_bc[i];
    }
    for (int i = lane; i < DD; i += 64) {
      hc[2 * AZ_DEP_EMB_ROWS + i] = p.q_b[i];
      hc[2 * AZ_DEP_EMB_ROWS + DD + i] = p.k_b[i];
    }
  }
  {
    float4 k0[KPL];
    load_consts(1, k0);
    store_consts(0, k0);
  }
  __syncthreads();

  // ---- stem: bf16 3x3 conv over 64 (padded) input channels, K = 576
  {
    constexpr int SSTEP = DNMB * 64 * 16;  // bytes per K step of the stem stream
    const uint8_t* sw8 = static_cast<const uint8_t*>(p.stem_w) + (size_t)lane * 16;
    f32x16 sacc[DNMB][NBW];
    // 36 K steps (tap = st / 4, 16 channels each): A fragments of step st in ring
    // slot st % 4, loaded three steps ahead; B fragments one step ahead
    constexpr int SR = 4, NST = 9 * DCP / 16;
    bf16x8 a[SR][DNMB];
    auto load_a = [&](int st) {
#pragma unroll
      for (int m = 0; m < DNMB; ++m) a[st % SR][m] = g_frag<MK_BF16>(sw8 + st * SSTEP + m * 64 * 16);
    };
    auto load_b = [&](int st, bf16x8(&dst)[NBW]) {
      const int tap = st / 4, cs = st % 4, dy = tap / 3 - 1, dx = tap % 3 - 1;
#pragma unroll
      for (int n = 0; n < NBW; ++n) {
        const int j = n * 32 + l32, r = (j >> 3) + dy, c = (j & 7) + dx;
        const bool ok = (unsigned)r < 8u && (unsigned)c < 8u;
        const int src = r * 8 + c;
        const int row = ok ? OFF_T + src * 128 : OFF_Z + ((src * 128) & 255);
        dst[n] = *reinterpret_cast<const bf16x8*>(smem + row + (((2 * cs + lhi) ^ swz128(src)) << 4));
      }
    };
#pragma unroll
    for (int st = 0; st < SR - 1; ++st) load_a(st);
    bf16x8 bcur[NBW], bnext[NBW];
    load_b(0, bcur);
#pragma unroll
    for (int st = 0; st < NST; ++st) {
      if (st + SR - 1 < NST) load_a(st + SR - 1);
      if (st + 1 < NST) load_b(st + 1, bnext);
#pragma unroll
      for (int m = 0; m < DNMB; ++m)
#pragma unroll
        for (int n = 0; n < NBW; ++n)
          sacc[m][n] = mma_bf16(a[st % SR][m], bcur[n], st == 0 ? f32x16{} : sacc[m][n]);
#pragma unroll
      for (int n = 0; n < NBW; ++n) bcur[n] = bnext[n];
    }
    // the tower's first weight steps, in flight during the stem's epilogue
    static_for<0, NBUF - 1>([&](auto i_c) {
      constexpr int i = decltype(i_c)::value;
      load_step(A[i], i * C::STEP_BYTES);
    });
    // epilogue: bias, activation (codes for int8), store in the tower format at OFF_H
#pragma unroll
    for (int m = 0; m < DNMB; ++m)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int ch0 = m * 32 + 8 * q + 4 * lhi;
        const float4 bb = *reinterpret_cast<const float4*>(p.bias + ch0);
        double mq[4] = {}, bq[4] = {};
        if constexpr (QUANT) {
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            mq[r] = p.qmul[ch0 + r];
            bq[r] = p.qbias[ch0 + r];
          }
        }
#pragma unroll
        for (int n = 0; n < NBW; ++n) {
          const int j = n * 32 + l32;
          const f32x16& v = sacc[m][n];
          if constexpr (!QUANT) {
            const float y0 = act_fn(v[4 * q + 0] + bb.x, cap), y1 = act_fn(v[4 * q + 1] + bb.y, cap);
            const float y2 = act_fn(v[4 * q + 2] + bb.z, cap), y3 = act_fn(v[4 * q + 3] + bb.w, cap);
            rlo[m][n][2 * q + 0] = pack_bf16x2(y0 - bf16_round(y0), y1 - bf16_round(y1));
            rlo[m][n][2 * q + 1] = pack_bf16x2(y2 - bf16_round(y2), y3 - bf16_round(y3));
            *reinterpret_cast<uint2*>(smem + OFF_H + j * RB + (R::pos(ch0 >> 3, R::sw(j)) << 4) + 8 * lhi) =
                make_uint2(pack_bf16x2(y0, y1), pack_bf16x2(y2, y3));
          } else {
            // fp32 sum of the bf16 matrix instruction; rescale and rounding in float64
            *reinterpret_cast<uint32_t*>(smem + OFF_H + j * RB + (R::pos(ch0 >> 4, R::sw(j)) << 4) + (ch0 & 15)) =
                pack_codes_d<MK>(__builtin_fma((double)v[4 * q + 0], mq[0], bq[0]),
                                 __builtin_fma((double)v[4 * q + 1], mq[1], bq[1]),
                                 __builtin_fma((double)v[4 * q + 2], mq[2], bq[2]),
                                 __builtin_fma((double)v[4 * q + 3], mq[3], bq[3]), p.qhi[0]);
          }
        }
      }
  }
  __syncthreads();

  // ---- residual tower
  {
    constexpr int CPT = C::CPT;
    acc_t c[DNMB][NBW];
    const int nconv = 2 * p.blocks;

    const int l32_ = l32, lhi_ = lhi;
    auto conv = [&](auto second_c, auto pool_c, auto lb_c, int n_conv) {
      constexpr bool SECOND = decltype(second_c)::value;
      constexpr bool POOL = decltype(pool_c)::value;   // first conv of a pooling block
      constexpr int LB = decltype(lb_c)::value;        // ring slot of the layer's first step
      // lane coordinates, opaque to the compiler per layer, so that the layer's
      // many lane-dependent addresses are computed in the layer instead of being
      // hoisted out of the block loop and held (or spilled) across it
      int l32 = l32_, lhi = lhi_;
      asm volatile("" : "+v"(l32), "+v"(lhi));
      const int wl = n_conv * (int)C::LAYER_BYTES;  // byte offset of the layer in the stream
      const bool has_next = n_conv + 1 < nconv;
      const int in_off = SECOND ? OFF_T : OFF_H;
      const int out_off = SECOND ? OFF_H : OFF_T;
      float* kslot = reinterpret_cast<float*>(smem + C::OFF_K + (n_conv & 1) * C::KSLOT);
      // the next layer's epilogue constants, in flight during this layer
      float4 kn[KPL];
      if (has_next) load_consts(n_conv + 2, kn);
      // B fragments of one K step.  Channel step cs reads logical chunk
      // lc = 2 cs + lhi of the tap's row, at chunk position (lc + rot) mod NC with
      // rot the row's rotation: from a per-tap base b0 = row + 16 (lhi + rot) the
      // address is b0 + 32 cs, except for the last steps, where lc + rot can pass
      // the row's end and the base is chosen per lane once per tap.
      constexpr int WRAP0 = (R::NC - 1 - R::RM) / 2;  // first step that can wrap
      constexpr int NWRAP = CPT > WRAP0 ? CPT - WRAP0 : 0;
      struct TapRows {
        int b0[NBW];
        int bw[NBW][NWRAP > 0 ? NWRAP : 1];
      };
      TapRows row, nrow;
      auto rows_for = [&](int tap, TapRows& tr) {
        const int dy = tap / 3 - 1, dx = tap % 3 - 1;
#pragma unroll
        for (int n = 0; n < NBW; ++n) {
          const int j = n * 32 + l32, r = (j >> 3) + dy, cc = (j & 7) + dx;
          const bool ok = (unsigned)r < 8u && (unsigned)cc < 8u;
          const int src = r * 8 + cc;
          const int ra = in_off + src * RB, rz = OFF_Z + ((src * RB) & 255);
          const int msk = -(int)ok;
          const int x = lhi + R::sw(src);
          tr.b0[n] = ((ra & msk) | (rz & ~msk)) + 16 * x;
#pragma unroll
          for (int k = 0; k < NWRAP; ++k)
            tr.bw[n][k] = tr.b0[n] - (2 * (WRAP0 + k) + x >= R::NC ? 16 * R::NC : 0);
        }
      };
      auto load_b = [&](const TapRows& tr, auto cs_c, frag_t(&dst)[NBW]) {
        constexpr int cs = decltype(cs_c)::value;
#pragma unroll
        for (int n = 0; n < NBW; ++n) {
          int base;
          if constexpr (cs >= WRAP0) base = tr.bw[n][cs - WRAP0];
          else base = tr.b0[n];
          dst[n] = *reinterpret_cast<const frag_t*>(smem + base + 32 * cs);
        }
      };
      frag_t bc[NBW], bn[NBW];
      rows_for(0, row);
      load_b(row, std::integral_constant<int, 0>{}, bc);

      // one tap: CPT K steps; R0 = ring slot of its first step
      auto tap_body = [&](auto r0_c, auto first_c, int tap) {
        constexpr int R0 = decltype(r0_c)::value;
        constexpr bool FIRST = decltype(first_c)::value;
        rows_for(tap + 1, nrow);
        static_for<0, CPT>([&](auto cs_c) {
          constexpr int cs = decltype(cs_c)::value;
          constexpr int cur = (R0 + cs) % NBUF;
          {
            // step tap*CPT + cs + NBUF-1 of this layer (of the next layer past its end;
            // past the network's last layer this layer is re-read and never used)
            const int gi = tap * CPT + cs + NBUF - 1;
            load_step(A[(cur + NBUF - 1) % NBUF], wl + ((has_next || gi < C::S) ? gi * C::STEP_BYTES : 0));
          }
          if constexpr (cs + 1 < CPT) load_b(row, std::integral_constant<int, cs + 1>{}, bn);
          else load_b(nrow, std::integral_constant<int, 0>{}, bn);
#pragma unroll
          for (int m = 0; m < DNMB; ++m)
#pragma unroll
            for (int n = 0; n < NBW; ++n)
              c[m][n] = T::mma(A[cur][m], bc[n], (FIRST && cs == 0) ? acc_t{} : c[m][n]);
#pragma unroll
          for (int n = 0; n < NBW; ++n) bc[n] = bn[n];
          // each MFMA followed by one of the next step's LDS reads, then by one of
          // the prefetched step's weight loads
          static_for<0, DNMB * 2>([&](auto i_c) {
            constexpr int i = decltype(i_c)::value;
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
            if constexpr (i < NBW) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            if constexpr (i < DNMB) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
          });
        });
        row = nrow;
      };
      constexpr int U = NBUF / gcd_c(CPT, NBUF), NIT = 8 / U, REM = 8 % U;
      tap_body(std::integral_constant<int, LB>{}, std::true_type{}, 0);
#pragma nounroll
      for (int it = 0; it < NIT; ++it) {
        static_for<0, U>([&](auto u_c) {
          constexpr int u = decltype(u_c)::value;
          tap_body(std::integral_constant<int, (LB + (1 + u) * CPT) % NBUF>{}, std::false_type{}, 1 + it * U + u);
        });
      }
      static_for<0, REM>([&](auto u_c) {
        constexpr int u = decltype(u_c)::value, t = 1 + NIT * U + u;
        tap_body(std::integral_constant<int, (LB + t * CPT) % NBUF>{}, std::false_type{}, t);
      });

      // global pooling: pooled channels' board mean and maximum, projected to a
      // context term that is folded into the regular channels' bias (in place in
      // this layer's constant slot)
      if constexpr (POOL) {
        // (1) the pooled channels to LDS as [pooled channel][square] in the T
        //     buffer (written by this layer's epilogue only afterwards); rows of
        //     256 bytes with 16-byte chunks XOR-swizzled by the row.  int8: the
        //     exact accumulators, activated in float64 in (2); bf16: act(acc + b1)
        float* pt = reinterpret_cast<float*>(smem + OFF_T);
        static_assert(DG * 64 * 4 <= C::BUF, "pooled activations fit in the T buffer");
        static_for<0, DNMB * 4>([&](auto k_c) {
          constexpr int k = decltype(k_c)::value, m = k / 4, q = k % 4;
          if constexpr (32 * m + 8 * q >= DFR) {
            const int ch0 = 32 * m + 8 * q + 4 * lhi;
            float4 bb = make_float4(0.f, 0.f, 0.f, 0.f);
            if constexpr (!QUANT) bb = *reinterpret_cast<const float4*>(kslot + ch0);
            const float bv[4] = {bb.x, bb.y, bb.z, bb.w};
#pragma unroll
            for (int r = 0; r < 4; ++r) {
              const int pc = ch0 + r - DFR;
#pragma unroll
              for (int n = 0; n < NBW; ++n) {
                const int sq = 32 * n + l32, idx = pc * 64 + (((sq >> 2) ^ (pc & 15)) << 2) + (sq & 3);
                if constexpr (QUANT) reinterpret_cast<int*>(pt)[idx] = (int)c[m][n][4 * q + r];
                else pt[idx] = med3(c[m][n][4 * q + r] + bv[r], 0.0f, cap);
              }
            }
          }
        });
        wave_lds_sync();
        // (2) lane pc < g: board sum (fp64) and maximum of its row; g = [mean, max]
        double* pg = reinterpret_cast<double*>(smem + C::OFF_PG);
        if (lane < DG) {
          const double2 mx_sum = pool_row<QUANT>(p, pt, lane, n_conv);
          pg[lane] = mx_sum.y * (1.0 / 64.0);
          pg[DG + lane] = mx_sum.x;
        }
        wave_lds_sync();
        // (3) c[o] = sum_i Wg[o][i] g[i] in fp64 (fp32 weights are exact): lane L
        //     takes outputs L and L + 64; the weights, [i/4][o][4] floats, stream
        //     in chunks of 16 inputs with the next chunk in flight
        const float4* wt = reinterpret_cast<const float4*>(p.pool_wt) +
                           (size_t)(n_conv / 2 / p.pool_every) * (2 * DG / 4) * AZ_DEP_POOL_OPAD;
        constexpr int NCH = 2 * DG / 16;
        float4 wbuf[2][2][4];
        auto load_chunk = [&](float4(&dst)[2][4], int chk) {
#pragma unroll
          for (int k4 = 0; k4 < 4; ++k4) {
            dst[0][k4] = wt[(size_t)(4 * chk + k4) * AZ_DEP_POOL_OPAD + lane];
            dst[1][k4] = wt[(size_t)(4 * chk + k4) * AZ_DEP_POOL_OPAD + 64 + lane];
          }
        };
        load_chunk(wbuf[0], 0);
        double c0 = 0.0, c1 = 0.0;
#pragma unroll
        for (int chk = 0; chk < NCH; ++chk) {
          if (chk + 1 < NCH) load_chunk(wbuf[(chk + 1) & 1], chk + 1);
#pragma unroll
          for (int k4 = 0; k4 < 4; ++k4) {
            const float4 w0 = wbuf[chk & 1][0][k4], w1 = wbuf[chk & 1][1][k4];
            const double* gi = pg + 16 * chk + 4 * k4;
            c0 = __builtin_fma((double)w0.x, gi[0], c0);
            c1 = __builtin_fma((double)w1.x, gi[0], c1);
            c0 = __builtin_fma((double)w0.y, gi[1], c0);
            c1 = __builtin_fma((double)w1.y, gi[1], c1);
            c0 = __builtin_fma((double)w0.z, gi[2], c0);
            c1 = __builtin_fma((double)w1.z, gi[2], c1);
            c0 = __builtin_fma((double)w0.w, gi[3], c0);
            c1 = __builtin_fma((double)w1.w, gi[3], c1);
          }
        }
        // regular channel o's bias takes c[o] (int8: in code units, c[o] / a[n+1])
        add_context<QUANT>(p, kslot, lane, c0, n_conv);
        if (lane + 64 < DFR) add_context<QUANT>(p, kslot, lane + 64, c1, n_conv);
        wave_lds_sync();
      }

      // epilogue: per run of 4 channels; LDS reads of constants (and residual
      // codes) issued two runs ahead
      float hi = 0.0f;
      double rq = 0.0;
      if constexpr (QUANT) {
        const double* kd = reinterpret_cast<const double*>(kslot);
        hi = (float)kd[2 * DF + 1];
        rq = SECOND ? kd[2 * DF] : 0.0;
      }
      constexpr int NRUN = DNMB * 4, EP_AHEAD = 2, EP_RING = EP_AHEAD + 1;
      constexpr bool RCODE = QUANT && SECOND;   // residual codes, read in place
      constexpr bool RHI = !QUANT && SECOND;    // residual hi parts, read in place
      // int8 constants: qbias and qmul of the run's four channels, float64
      struct KQ { double b[4], m[4]; };
      float4 kb[QUANT ? 1 : EP_RING];
      KQ kq[QUANT ? EP_RING : 1];
      uint32_t rcode[RCODE ? EP_RING : 1][NBW];
      uint2 rhi[RHI ? EP_RING : 1][NBW];
      auto ep_addr = [&](int m, int q, int n) {
        const int j = n * 32 + l32;
        const int ch0 = m * 32 + 8 * q + 4 * lhi;
        const int rowo = out_off + j * RB;
        if constexpr (QUANT) return rowo + (R::pos(ch0 >> 4, R::sw(j)) << 4) + (ch0 & 15);
        else return rowo + (R::pos(ch0 >> 3, R::sw(j)) << 4) + 8 * lhi;
      };
      auto ep_load = [&](auto k_c) {
        constexpr int k = decltype(k_c)::value, m = k / 4, q = k % 4, slot = k % EP_RING;
        const int ch0 = m * 32 + 8 * q + 4 * lhi;
        if constexpr (QUANT) {
          const double* kd = reinterpret_cast<const double*>(kslot);
#pragma unroll
          for (int r = 0; r < 4; r += 2) {
            const double2 b2 = *reinterpret_cast<const double2*>(kd + ch0 + r);
            const double2 m2 = *reinterpret_cast<const double2*>(kd + DF + ch0 + r);
            kq[slot].b[r] = b2.x;
            kq[slot].b[r + 1] = b2.y;
            kq[slot].m[r] = m2.x;
            kq[slot].m[r + 1] = m2.y;
          }
        } else {
          kb[slot] = *reinterpret_cast<const float4*>(kslot + ch0);
        }
        if constexpr (RCODE) {
#pragma unroll
          for (int n = 0; n < NBW; ++n) rcode[slot][n] = *reinterpret_cast<const uint32_t*>(smem + ep_addr(m, q, n));
        }
        if constexpr (RHI) {
#pragma unroll
          for (int n = 0; n < NBW; ++n) rhi[slot][n] = *reinterpret_cast<const uint2*>(smem + ep_addr(m, q, n));
        }
      };
      static_for<0, EP_AHEAD>([&](auto k_c) { ep_load(k_c); });
      static_for<0, NRUN>([&](auto k_c) {
        constexpr int k = decltype(k_c)::value, m = k / 4, q = k % 4, slot = k % EP_RING;
        if constexpr (k + EP_AHEAD < NRUN) ep_load(std::integral_constant<int, k + EP_AHEAD>{});
#pragma unroll
        for (int n = 0; n < NBW; ++n) {
          const int addr = ep_addr(m, q, n);
          const acc_t& v = c[m][n];
          if constexpr (!QUANT) {
            const float4 bb = kb[slot];
            float y0 = v[4 * q + 0] + bb.x, y1 = v[4 * q + 1] + bb.y;
            float y2 = v[4 * q + 2] + bb.z, y3 = v[4 * q + 3] + bb.w;
            if constexpr (SECOND) {
              // block input h = hi + lo (exact in fp32)
              const uint2 hv = rhi[slot][n];
              const uint32_t l01 = rlo[m][n][2 * q], l23 = rlo[m][n][2 * q + 1];
              y0 = act_fn(y0 + (__uint_as_float(hv.x << 16) + __uint_as_float(l01 << 16)), cap);
              y1 = act_fn(y1 + (__uint_as_float(hv.x & 0xffff0000u) + __uint_as_float(l01 & 0xffff0000u)), cap);
              y2 = act_fn(y2 + (__uint_as_float(hv.y << 16) + __uint_as_float(l23 << 16)), cap);
              y3 = act_fn(y3 + (__uint_as_float(hv.y & 0xffff0000u) + __uint_as_float(l23 & 0xffff0000u)), cap);
              rlo[m][n][2 * q + 0] = pack_bf16x2(y0 - bf16_round(y0), y1 - bf16_round(y1));
              rlo[m][n][2 * q + 1] = pack_bf16x2(y2 - bf16_round(y2), y3 - bf16_round(y3));
            } else {
              y0 = act_fn(y0, cap);
              y1 = act_fn(y1, cap);
              y2 = act_fn(y2, cap);
              y3 = act_fn(y3, cap);
            }
            *reinterpret_cast<uint2*>(smem + addr) = make_uint2(pack_bf16x2(y0, y1), pack_bf16x2(y2, y3));
          } else {
            // float64 requantisation: z = acc * qmul + qbias (+ residual code * qres)
            const KQ& kk = kq[slot];
            double z[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) z[r] = __builtin_fma((double)v[4 * q + r], kk.m[r], kk.b[r]);
            if constexpr (SECOND) {
              const uint32_t rc = rcode[slot][n];
              z[0] = __builtin_fma(code_value_d<MK, 0>(rc), rq, z[0]);
              z[1] = __builtin_fma(code_value_d<MK, 1>(rc), rq, z[1]);
              z[2] = __builtin_fma(code_value_d<MK, 2>(rc), rq, z[2]);
              z[3] = __builtin_fma(code_value_d<MK, 3>(rc), rq, z[3]);
            }
            *reinterpret_cast<uint32_t*>(smem + addr) = pack_codes_d<MK>(z[0], z[1], z[2], z[3], hi);
          }
        }
      });
      if (has_next) store_consts((n_conv + 1) & 1, kn);
      __syncthreads();
    };

    for (int blk = 0; blk < p.blocks; ++blk) {
      const bool pool = p.pool_every > 0 && blk % p.pool_every == p.pool_every - 1;
      if (pool) conv(std::false_type{}, std::true_type{}, std::integral_constant<int, 0>{}, 2 * blk);
      else conv(std::false_type{}, std::false_type{}, std::integral_constant<int, 0>{}, 2 * blk);
      conv(std::true_type{}, std::false_type{}, std::integral_constant<int, C::S % NBUF>{}, 2 * blk + 1);
    }
  }

  // ---- heads input (bf16 networks): the low part h - bf16(h) of the fp32
  // residual as bf16 rows [square][F] at OFF_X, H holding bf16(h); int8
  // networks read the final codes from H and convert them in registers
  using RX = Rot<C::RBX>;
  if constexpr (!QUANT) {
#pragma unroll
    for (int m = 0; m < DNMB; ++m)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int ch0 = m * 32 + 8 * q + 4 * lhi;
#pragma unroll
        for (int n = 0; n < NBW; ++n) {
          const int j = n * 32 + l32;
          *reinterpret_cast<uint2*>(smem + C::OFF_X + j * C::RBX + (RX::pos(ch0 >> 3, RX::sw(j)) << 4) + 8 * lhi) =
              make_uint2(rlo[m][n][2 * q], rlo[m][n][2 * q + 1]);
        }
      }
  }
  __syncthreads();

  dep_heads<MK>(p, smem, legal, policy, value, wdl, b, lane);
}

template <int MK>
__global__ __attribute__((amdgpu_flat_work_group_size(256, 256), amdgpu_waves_per_eu(1, 1))) void
az_dep_kernel4(AzDevNet p, const float* __restrict__ planes, const uint8_t* __restrict__ legal,
              float* __restrict__ policy, float* __restrict__ value, float* __restrict__ wdl) {
  using C = DepCfg<MK>;
  using T = typename C::T;
  using frag_t = typename T::frag;
  using acc_t = typename T::acc;
  using R = Rot<C::RB>;
  constexpr bool QUANT = C::QUANT;
  constexpr int RB = C::RB, OFF_H = C::OFF_H, OFF_T = C::OFF_T, OFF_Z = C::OFF_Z;

  __shared__ __attribute__((aligned(16))) uint8_t smem[C::SMEM4];

  // Tiles of a layer: five 32-channel blocks x two half-board square blocks.
  // Wave w (one per SIMD) owns both tiles of block w, and waves 0 and 1 also
  // tile (4, w), so no SIMD runs more than three of the ten MFMA chains of a K
  // step.
  constexpr int NWB = 4;                     // waves per board
  static_assert(DNMB == NWB + 1, "four waves, five blocks");
  constexpr int NT = 64 * NWB;
  constexpr int MBW = 1;                     // blocks whose two tiles the wave owns
  constexpr int NBW = 2;                     // half-board square blocks
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l32 = lane & 31, lhi = lane >> 5;
  const int mb0 = wave;                      // first block the wave owns
  const int b = blockIdx.x;
  const int Cin = p.in_planes;
  const float cap = p.act_cap;

  // ---- ingest: zero region, planes -> bf16 [square][64 channels] at OFF_T
  for (int i = tid; i < C::ZB / 16; i += NT)
    *reinterpret_cast<i32x4*>(smem + OFF_Z + i * 16) = i32x4{0, 0, 0, 0};
  {
    // item k = planes 8k..8k+7 (items wave, wave + NWB, ...): lane = square,
    // eight coalesced loads, one 16-byte store
    constexpr int KI = DCP / 8, KW = KI / NWB;
    static_assert(KI % NWB == 0, "ingest items per wave");
    float pv[KW][8];
#pragma unroll
    for (int kw = 0; kw < KW; ++kw)
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const int c = 8 * (wave + NWB * kw) + t;
        const bool ok = c < Cin;
        const float x = planes[((size_t)b * Cin + (ok ? c : 0)) * 64 + lane];
        pv[kw][t] = ok ? x : 0.0f;
      }
#pragma unroll
    for (int kw = 0; kw < KW; ++kw) {
      const int k = wave + NWB * kw;
      *reinterpret_cast<uint4*>(smem + OFF_T + lane * 128 + ((k ^ swz128(lane)) << 4)) =
          make_uint4(pack_bf16x2(pv[kw][0], pv[kw][1]), pack_bf16x2(pv[kw][2], pv[kw][3]),
                     pack_bf16x2(pv[kw][4], pv[kw][5]), pack_bf16x2(pv[kw][6], pv[kw][7]));
    }
  }

  // tower weight stream, read through a buffer resource: the lane's offsets
  // (its own block, and block 4) are constant VGPRs, a step's byte offset is a
  // scalar and a block's a literal, so the loads cost no vector address
  // arithmetic.  K step i of the stream lives in ring slot i % NBUF, loaded
  // NBUF - 1 steps ahead: a wave's K step is two or three MFMAs, so the ring is
  // deep enough to cover a load from L2 or the Infinity Cache (int8 15 steps,
  // bf16 10: measured best among the depths that tile two layers).
  constexpr int NBUF = QUANT ? 15 : 10;
  static_assert((2 * C::S) % NBUF == 0, "every block's first conv starts at ring slot 0");
  const __amdgpu_buffer_rsrc_t twr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<void*>(p.tower_w), (short)0, (int)(2 * p.blocks * C::LAYER_BYTES), 0x00020000);
  const int tvoff = (mb0 * 64 + lane) * T::FB;
  const int tvoffx = ((DNMB - 1) * 64 + lane) * T::FB;
  // per-layer epilogue constants of conv index k (0 = stem): [bias F] floats, or
  // [qbias F | qmul F] doubles, as thread-held 16-byte chunks loaded at the start
  // of a layer and parked in LDS before its barrier
  constexpr int KV = C::KSLOT / 16;                  // 16-byte chunks per slot
  constexpr int KPL = (KV + NT - 1) / NT;            // per thread
  auto load_consts = [&](int k, float4(&dst)[KPL]) {
#pragma unroll
    for (int t = 0; t < KPL; ++t) {
      const int i = tid + NT * t;
      const void* src;
      if constexpr (QUANT)
        src = i < DF / 2 ? p.qbias + (size_t)k * DF + 2 * i
              : i < DF   ? p.qmul + (size_t)k * DF + 2 * (i - DF / 2)
                         : p.qext + 2 * (size_t)k;
      else src = p.bias + (size_t)k * DF + 4 * i;
      dst[t] = i < KV ? *reinterpret_cast<const float4*>(src) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  };
  auto store_consts = [&](int slot, const float4(&v)[KPL]) {
    float4* dst = reinterpret_cast<float4*>(smem + C::OFF_K + slot * C::KSLOT);
#pragma unroll
    for (int t = 0; t < KPL; ++t)
      if (tid + NT * t < KV) dst[tid + NT * t] = v[t];
  };
  // head constants, staged once: embedding row scale and bias, query and key biases
  {
    float* hc = reinterpret_cast<float*>(smem + C::OFF_HC);
    for (int i = tid; i < AZ_DEP_EMB_ROWS; i += NT) {
      hc[i] = p.emb_sc[i];
      hc[AZ_DEP_EMB_ROWS + i] = p.emb_bc[i];
    }
    for (int i = tid; i < DD; i += NT) {
      hc[2 * AZ_DEP_EMB_ROWS + i] = p.q_b[i];
      hc[2 * AZ_DEP_EMB_ROWS + DD + i] = p.k_b[i];
    }
  }
  {
    float4 k0[KPL];
    load_consts(1, k0);
    store_consts(0, k0);
  }

  // ---- stem and tower of one wave.  XN >= 0: the wave also owns tile (4, XN).
  // Fragment / accumulator set m < MBW is block mb0 + m (both tiles); set MBW,
  // when present, is block 4 (tile XN only).  Every wave meets the same
  // sequence of workgroup barriers.
  // int8 layers without pooling move the epilogue of tile (4, n) from wave n to
  // wave 2 + n (MV = n), which finishes its K loop earlier; the tile's
  // accumulators go through LDS.
  constexpr bool MOVE = QUANT;
  auto trunk = [&](auto xn_c, auto mv_c) {
    constexpr int XN = decltype(xn_c)::value;
    constexpr int MV = decltype(mv_c)::value;      // tile (4, MV)'s moved epilogue (waves 2, 3)
    constexpr int NAF = MBW + (XN >= 0 ? 1 : 0);   // weight fragments per K step
    auto blk_of = [&](int m) { return m < MBW ? mb0 + m : DNMB - 1; };
    auto n_lo = [](int m) constexpr { return m < MBW ? 0 : (XN >= 0 ? XN : MV); };
    auto n_hi = [](int m) constexpr { return m < MBW ? NBW : (XN >= 0 ? XN : MV) + 1; };

    // residual stream of the board (bf16 networks): h = hi + lo, hi = bf16(h) in
    // the H buffer (the convolution operand), lo = bf16(h - hi) packed here, two
    // per register: [set][half][run of 4 channels][2]
    uint32_t rlo[QUANT ? 1 : NAF][QUANT ? 1 : NBW][QUANT ? 1 : 8];

    frag_t A[NBUF][NAF];
    auto load_step = [&](frag_t(&dst)[NAF], int soff) {
#pragma unroll
      for (int m = 0; m < MBW; ++m)
        dst[m] = __builtin_bit_cast(frag_t, __builtin_amdgcn_raw_buffer_load_b128(twr, tvoff, soff + m * 64 * T::FB, 0));
      if constexpr (NAF > MBW)
        dst[MBW] = __builtin_bit_cast(frag_t, __builtin_amdgcn_raw_buffer_load_b128(twr, tvoffx, soff, 0));
    };

    // ---- stem: bf16 3x3 conv over 64 (padded) input channels, K = 576
    {
      constexpr int SSTEP = DNMB * 64 * 16;  // bytes per K step of the stem stream
      const uint8_t* sw8 = static_cast<const uint8_t*>(p.stem_w) + (size_t)lane * 16;
      f32x16 sacc[NAF][NBW];
      // 36 K steps (tap = st / 4, 16 channels each): A fragments of step st in ring
      // slot st % 12, loaded eleven steps ahead, the first ones before the ingest
      // barrier; B fragments one step ahead
      constexpr int SR = 12, NST = 9 * DCP / 16;
      bf16x8 a[SR][NAF];
      auto load_a = [&](int st) {
#pragma unroll
        for (int m = 0; m < NAF; ++m) a[st % SR][m] = g_frag<MK_BF16>(sw8 + st * SSTEP + blk_of(m) * 64 * 16);
      };
      auto load_b = [&](int st, bf16x8(&dst)[NBW]) {
        const int tap = st / 4, cs = st % 4, dy = tap / 3 - 1, dx = tap % 3 - 1;
#pragma unroll
        for (int n = 0; n < NBW; ++n) {
          const int j = n * 32 + l32, r = (j >> 3) + dy, c = (j & 7) + dx;
          const bool ok = (unsigned)r < 8u && (unsigned)c < 8u;
          const int src = r * 8 + c;
          const int row = ok ? OFF_T + src * 128 : OFF_Z + ((src * 128) & 255);
          dst[n] = *reinterpret_cast<const bf16x8*>(smem + row + (((2 * cs + lhi) ^ swz128(src)) << 4));
        }
      };
#pragma unroll
      for (int st = 0; st < SR - 1; ++st) load_a(st);
      __syncthreads();  // the ingest's planes and constants are in LDS
      bf16x8 bcur[NBW], bnext[NBW];
      load_b(0, bcur);
#pragma unroll
      for (int st = 0; st < NST; ++st) {
        if (st + SR - 1 < NST) load_a(st + SR - 1);
        if (st + 1 < NST) load_b(st + 1, bnext);
#pragma unroll
        for (int m = 0; m < NAF; ++m)
#pragma unroll
          for (int n = n_lo(m); n < n_hi(m); ++n)
            sacc[m][n] = mma_bf16(a[st % SR][m], bcur[n], st == 0 ? f32x16{} : sacc[m][n]);
#pragma unroll
        for (int n = 0; n < NBW; ++n) bcur[n] = bnext[n];
      }
      // the tower's first weight steps, in flight during the stem's epilogue
      static_for<0, NBUF - 1>([&](auto i_c) {
        constexpr int i = decltype(i_c)::value;
        load_step(A[i], i * C::STEP_BYTES);
      });
      // epilogue: bias, activation (codes for int8), store in the tower format at OFF_H
#pragma unroll
      for (int m = 0; m < NAF; ++m)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int ch0 = blk_of(m) * 32 + 8 * q + 4 * lhi;
          const float4 bb = *reinterpret_cast<const float4*>(p.bias + ch0);
          double mq[4] = {}, bq[4] = {};
          if constexpr (QUANT) {
  #pragma unroll
            for (int r = 0; r < 4; ++r) {
              mq[r] = p.qmul[ch0 + r];
              bq[r] = p.qbias[ch0 + r];
            }
          }
#pragma unroll
          for (int n = n_lo(m); n < n_hi(m); ++n) {
            const int j = n * 32 + l32;
            const f32x16& v = sacc[m][n];
            if constexpr (!QUANT) {
              const float y0 = act_fn(v[4 * q + 0] + bb.x, cap), y1 = act_fn(v[4 * q + 1] + bb.y, cap);
              const float y2 = act_fn(v[4 * q + 2] + bb.z, cap), y3 = act_fn(v[4 * q + 3] + bb.w, cap);
              rlo[m][n][2 * q + 0] = pack_bf16x2(y0 - bf16_round(y0), y1 - bf16_round(y1));
              rlo[m][n][2 * q + 1] = pack_bf16x2(y2 - bf16_round(y2), y3 - bf16_round(y3));
              *reinterpret_cast<uint2*>(smem + OFF_H + j * RB + (R::pos(ch0 >> 3, R::sw(j)) << 4) + 8 * lhi) =
                  make_uint2(pack_bf16x2(y0, y1), pack_bf16x2(y2, y3));
            } else {
              // fp32 sum of the bf16 matrix instruction; rescale and rounding in float64
              *reinterpret_cast<uint32_t*>(smem + OFF_H + j * RB + (R::pos(ch0 >> 4, R::sw(j)) << 4) + (ch0 & 15)) =
                  pack_codes_d<MK>(__builtin_fma((double)v[4 * q + 0], mq[0], bq[0]),
                                   __builtin_fma((double)v[4 * q + 1], mq[1], bq[1]),
                                   __builtin_fma((double)v[4 * q + 2], mq[2], bq[2]),
                                   __builtin_fma((double)v[4 * q + 3], mq[3], bq[3]), p.qhi[0]);
            }
          }
        }
    }
    __syncthreads();

    // ---- residual tower
    {
      constexpr int CPT = C::CPT;
      acc_t c[MBW + 1][NBW];
      const int nconv = 2 * p.blocks;

      const int l32_ = l32, lhi_ = lhi;
      auto conv = [&](auto second_c, auto pool_c, auto lb_c, int n_conv) {
        constexpr bool SECOND = decltype(second_c)::value;
        constexpr bool POOL = decltype(pool_c)::value;   // first conv of a pooling block
        constexpr int LB = decltype(lb_c)::value;        // ring slot of the layer's first step
        // lane coordinates, opaque to the compiler per layer, so that the layer's
        // many lane-dependent addresses are computed in the layer instead of being
        // hoisted out of the block loop and held (or spilled) across it
        int l32 = l32_, lhi = lhi_;
        asm volatile("" : "+v"(l32), "+v"(lhi));
        const int wl = n_conv * (int)C::LAYER_BYTES;  // byte offset of the layer in the stream
        const bool has_next = n_conv + 1 < nconv;
        const int in_off = SECOND ? OFF_T : OFF_H;
        const int out_off = SECOND ? OFF_H : OFF_T;
        float* kslot = reinterpret_cast<float*>(smem + C::OFF_K + (n_conv & 1) * C::KSLOT);
        // the next layer's epilogue constants, in flight during this layer
        float4 kn[KPL];
        if (has_next) load_consts(n_conv + 2, kn);
        // a pooling layer's projection weights (waves 0 and 1: output 64 wave +
        // lane, all 2g inputs as [i/4] float4s), in flight during the K loop
        constexpr int NWP = POOL ? 2 * DG / 4 : 1;
        float4 wpool[NWP];
        if constexpr (POOL) {
          const float4* wt = reinterpret_cast<const float4*>(p.pool_wt) +
                             (size_t)(n_conv / 2 / p.pool_every) * (2 * DG / 4) * AZ_DEP_POOL_OPAD + 64 * (wave & 1) + lane;
#pragma unroll
          for (int i4 = 0; i4 < NWP; ++i4) wpool[i4] = wt[(size_t)i4 * AZ_DEP_POOL_OPAD];
        }
        // B fragments of one K step.  Channel step cs reads logical chunk
        // lc = 2 cs + lhi of the tap's row, at chunk position (lc + rot) mod NC with
        // rot the row's rotation: from a per-tap base b0 = row + 16 (lhi + rot) the
        // address is b0 + 32 cs, except for the last steps, where lc + rot can pass
        // the row's end and the base is chosen per lane once per tap.
        constexpr int WRAP0 = (R::NC - 1 - R::RM) / 2;  // first step that can wrap
        constexpr int NWRAP = CPT > WRAP0 ? CPT - WRAP0 : 0;
        struct TapRows {
          int b0[NBW];
          int bw[NBW][NWRAP > 0 ? NWRAP : 1];
        };
        TapRows row, nrow;
        auto rows_for = [&](int tap, TapRows& tr) {
          const int dy = tap / 3 - 1, dx = tap % 3 - 1;
#pragma unroll
          for (int n = 0; n < NBW; ++n) {
            const int j = n * 32 + l32, r = (j >> 3) + dy, cc = (j & 7) + dx;
            const bool ok = (unsigned)r < 8u && (unsigned)cc < 8u;
            const int src = r * 8 + cc;
            const int ra = in_off + src * RB, rz = OFF_Z + ((src * RB) & 255);
            const int msk = -(int)ok;
            const int x = lhi + R::sw(src);
            tr.b0[n] = ((ra & msk) | (rz & ~msk)) + 16 * x;
#pragma unroll
            for (int k = 0; k < NWRAP; ++k)
              tr.bw[n][k] = tr.b0[n] - (2 * (WRAP0 + k) + x >= R::NC ? 16 * R::NC : 0);
          }
        };
        auto load_b = [&](const TapRows& tr, auto cs_c, frag_t(&dst)[NBW]) {
          constexpr int cs = decltype(cs_c)::value;
#pragma unroll
          for (int n = 0; n < NBW; ++n) {
            int base;
            if constexpr (cs >= WRAP0) base = tr.bw[n][cs - WRAP0];
            else base = tr.b0[n];
            dst[n] = *reinterpret_cast<const frag_t*>(smem + base + 32 * cs);
          }
        };
        frag_t bc[NBW], bn[NBW];
        rows_for(0, row);
        load_b(row, std::integral_constant<int, 0>{}, bc);

        // one tap: CPT K steps; R0 = ring slot of its first step
        auto tap_body = [&](auto r0_c, auto first_c, int tap) {
          constexpr int R0 = decltype(r0_c)::value;
          constexpr bool FIRST = decltype(first_c)::value;
          rows_for(tap + 1, nrow);
          static_for<0, CPT>([&](auto cs_c) {
            constexpr int cs = decltype(cs_c)::value;
            constexpr int cur = (R0 + cs) % NBUF;
            {
              // step tap*CPT + cs + NBUF-1 of this layer (of the next layer past its end;
              // past the network's last layer this layer is re-read and never used)
              const int gi = tap * CPT + cs + NBUF - 1;
              load_step(A[(cur + NBUF - 1) % NBUF], wl + ((has_next || gi < C::S) ? gi * C::STEP_BYTES : 0));
            }
            if constexpr (cs + 1 < CPT) load_b(row, std::integral_constant<int, cs + 1>{}, bn);
            else load_b(nrow, std::integral_constant<int, 0>{}, bn);
#pragma unroll
            for (int m = 0; m < NAF; ++m)
#pragma unroll
              for (int n = n_lo(m); n < n_hi(m); ++n)
                c[m][n] = T::mma(A[cur][m], bc[n], (FIRST && cs == 0) ? acc_t{} : c[m][n]);
#pragma unroll
            for (int n = 0; n < NBW; ++n) bc[n] = bn[n];
            // each MFMA followed by one of the next step's LDS reads, then by one of
            // the prefetched step's weight loads
            static_for<0, MBW * NBW + NAF - MBW>([&](auto i_c) {
              constexpr int i = decltype(i_c)::value;
              __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
              if constexpr (i < NBW) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
              if constexpr (i < NAF) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
            });
          });
          row = nrow;
        };
        constexpr int U = NBUF / gcd_c(CPT, NBUF), NIT = 8 / U, REM = 8 % U;
        tap_body(std::integral_constant<int, LB>{}, std::true_type{}, 0);
#pragma nounroll
        for (int it = 0; it < NIT; ++it) {
          static_for<0, U>([&](auto u_c) {
            constexpr int u = decltype(u_c)::value;
            tap_body(std::integral_constant<int, (LB + (1 + u) * CPT) % NBUF>{}, std::false_type{}, 1 + it * U + u);
          });
        }
        static_for<0, REM>([&](auto u_c) {
          constexpr int u = decltype(u_c)::value, t = 1 + NIT * U + u;
          tap_body(std::integral_constant<int, (LB + t * CPT) % NBUF>{}, std::false_type{}, t);
        });

        // global pooling: pooled channels' board mean and maximum, projected to a
        // context term that is folded into the regular channels' bias (in place in
        // this layer's constant slot)
        if constexpr (POOL) {
          // (1) the pooled channels to LDS as [pooled channel][square] in the T
          //     buffer (written by this layer's epilogue only afterwards); rows of
          //     256 bytes with 16-byte chunks XOR-swizzled by the row.  int8: the
          //     exact accumulators, activated in float64 in (2); bf16: act(acc + b1)
          float* pt = reinterpret_cast<float*>(smem + OFF_T);
          static_assert(DG * 64 * 4 <= C::BUF, "pooled activations fit in the T buffer");
          static_for<0, NAF * 4>([&](auto k_c) {
            constexpr int k = decltype(k_c)::value, m = k / 4, q = k % 4;
            if (32 * blk_of(m) + 8 * q >= DFR) {
              const int ch0 = 32 * blk_of(m) + 8 * q + 4 * lhi;
              float4 bb = make_float4(0.f, 0.f, 0.f, 0.f);
              if constexpr (!QUANT) bb = *reinterpret_cast<const float4*>(kslot + ch0);
              const float bv[4] = {bb.x, bb.y, bb.z, bb.w};
#pragma unroll
              for (int r = 0; r < 4; ++r) {
                const int pc = ch0 + r - DFR;
#pragma unroll
                for (int n = n_lo(m); n < n_hi(m); ++n) {
                  const int sq = 32 * n + l32, idx = pc * 64 + (((sq >> 2) ^ (pc & 15)) << 2) + (sq & 3);
                  if constexpr (QUANT) reinterpret_cast<int*>(pt)[idx] = (int)c[m][n][4 * q + r];
                  else pt[idx] = med3(c[m][n][4 * q + r] + bv[r], 0.0f, cap);
                }
              }
            }
          });
          wave_lds_sync();
          // (2) wave w, lane l < g/4: board sum (fp64) and maximum of row
          //     pc = g/4 w + l; g = [mean, max]
          double* pg = reinterpret_cast<double*>(smem + C::OFF_PG);
          static_assert(DG % 4 == 0, "pooled rows per wave");
          if (lane < DG / 4) {
            const int pc = (DG / 4) * wave + lane;
            const double2 mx_sum = pool_row<QUANT>(p, pt, pc, n_conv);
            pg[pc] = mx_sum.y * (1.0 / 64.0);
            pg[DG + pc] = mx_sum.x;
          }
          wave_lds_sync();
          // (3) c[o] = sum_i Wg[o][i] g[i] in fp64 (fp32 weights are exact): waves 0
          //     and 1 take output 64 wave + lane with the prefetched weights
          if (wave < 2) {
            const int o = 64 * wave + lane;
            double co = 0.0;
#pragma unroll
            for (int i4 = 0; i4 < NWP; ++i4) {
              const float4 w = wpool[i4];
              const double* gi = pg + 4 * i4;
              co = __builtin_fma((double)w.x, gi[0], co);
              co = __builtin_fma((double)w.y, gi[1], co);
              co = __builtin_fma((double)w.z, gi[2], co);
              co = __builtin_fma((double)w.w, gi[3], co);
            }
            // regular channel o's bias takes c[o] (int8: in code units, c[o] / a[n+1])
            if (o < DFR) add_context<QUANT>(p, kslot, o, co, n_conv);
          }
          wave_lds_sync();
        }

        // epilogue: per run of 4 channels; LDS reads of constants (and residual
        // codes) issued two runs ahead
        float hi = 0.0f;
        double rq = 0.0;
        if constexpr (QUANT) {
          const double* kd = reinterpret_cast<const double*>(kslot);
          hi = (float)kd[2 * DF + 1];
          rq = SECOND ? kd[2 * DF] : 0.0;
        }
        constexpr int EP_AHEAD = 2, EP_RING = EP_AHEAD + 1;
        constexpr bool RCODE = QUANT && SECOND;   // residual codes, read in place
        constexpr bool RHI = !QUANT && SECOND;    // residual hi parts, read in place
        // int8 constants: qbias and qmul of the run's four channels, float64
        struct KQ { double b[4], m[4]; };
        float4 kb[QUANT ? 1 : EP_RING];
        KQ kq[QUANT ? EP_RING : 1];
        uint32_t rcode[RCODE ? EP_RING : 1][NBW];
        uint2 rhi[RHI ? EP_RING : 1][NBW];
        auto ep_addr = [&](int m, int q, int n) {
          const int j = n * 32 + l32;
          const int ch0 = blk_of(m) * 32 + 8 * q + 4 * lhi;
          const int rowo = out_off + j * RB;
          if constexpr (QUANT) return rowo + (R::pos(ch0 >> 4, R::sw(j)) << 4) + (ch0 & 15);
          else return rowo + (R::pos(ch0 >> 3, R::sw(j)) << 4) + 8 * lhi;
        };
        auto ep_load = [&](auto k_c) {
          constexpr int k = decltype(k_c)::value, m = k / 4, q = k % 4, slot = k % EP_RING;
          const int ch0 = blk_of(m) * 32 + 8 * q + 4 * lhi;
          if constexpr (QUANT) {
            const double* kd = reinterpret_cast<const double*>(kslot);
  #pragma unroll
            for (int r = 0; r < 4; r += 2) {
              const double2 b2 = *reinterpret_cast<const double2*>(kd + ch0 + r);
              const double2 m2 = *reinterpret_cast<const double2*>(kd + DF + ch0 + r);
              kq[slot].b[r] = b2.x;
              kq[slot].b[r + 1] = b2.y;
              kq[slot].m[r] = m2.x;
              kq[slot].m[r + 1] = m2.y;
            }
          } else {
            kb[slot] = *reinterpret_cast<const float4*>(kslot + ch0);
          }
          if constexpr (RCODE) {
#pragma unroll
            for (int n = n_lo(m); n < n_hi(m); ++n) rcode[slot][n] = *reinterpret_cast<const uint32_t*>(smem + ep_addr(m, q, n));
          }
          if constexpr (RHI) {
#pragma unroll
            for (int n = n_lo(m); n < n_hi(m); ++n) rhi[slot][n] = *reinterpret_cast<const uint2*>(smem + ep_addr(m, q, n));
          }
        };
        // runs [K0, K1) (run k: set k / 4, channels 8 (k % 4) .. of the set's block)
        auto epi_runs = [&](auto k0_c, auto k1_c) {
        constexpr int K0 = decltype(k0_c)::value, K1 = decltype(k1_c)::value;
        static_for<K0, (K0 + EP_AHEAD < K1 ? K0 + EP_AHEAD : K1)>([&](auto k_c) { ep_load(k_c); });
        static_for<K0, K1>([&](auto k_c) {
          constexpr int k = decltype(k_c)::value, m = k / 4, q = k % 4, slot = k % EP_RING;
          if constexpr (k + EP_AHEAD < K1) ep_load(std::integral_constant<int, k + EP_AHEAD>{});
#pragma unroll
          for (int n = n_lo(m); n < n_hi(m); ++n) {
            const int addr = ep_addr(m, q, n);
            const acc_t& v = c[m][n];
            if constexpr (!QUANT) {
              const float4 bb = kb[slot];
              float y0 = v[4 * q + 0] + bb.x, y1 = v[4 * q + 1] + bb.y;
              float y2 = v[4 * q + 2] + bb.z, y3 = v[4 * q + 3] + bb.w;
              if constexpr (SECOND) {
                // block input h = hi + lo (exact in fp32)
                const uint2 hv = rhi[slot][n];
                const uint32_t l01 = rlo[m][n][2 * q], l23 = rlo[m][n][2 * q + 1];
                y0 = act_fn(y0 + (__uint_as_float(hv.x << 16) + __uint_as_float(l01 << 16)), cap);
                y1 = act_fn(y1 + (__uint_as_float(hv.x & 0xffff0000u) + __uint_as_float(l01 & 0xffff0000u)), cap);
                y2 = act_fn(y2 + (__uint_as_float(hv.y << 16) + __uint_as_float(l23 << 16)), cap);
                y3 = act_fn(y3 + (__uint_as_float(hv.y & 0xffff0000u) + __uint_as_float(l23 & 0xffff0000u)), cap);
                rlo[m][n][2 * q + 0] = pack_bf16x2(y0 - bf16_round(y0), y1 - bf16_round(y1));
                rlo[m][n][2 * q + 1] = pack_bf16x2(y2 - bf16_round(y2), y3 - bf16_round(y3));
              } else {
                y0 = act_fn(y0, cap);
                y1 = act_fn(y1, cap);
                y2 = act_fn(y2, cap);
                y3 = act_fn(y3, cap);
              }
              *reinterpret_cast<uint2*>(smem + addr) = make_uint2(pack_bf16x2(y0, y1), pack_bf16x2(y2, y3));
            } else {
              // float64 requantisation: z = acc * qmul + qbias (+ residual code * qres)
              const KQ& kk = kq[slot];
              double z[4];
  #pragma unroll
              for (int r = 0; r < 4; ++r) z[r] = __builtin_fma((double)v[4 * q + r], kk.m[r], kk.b[r]);
              if constexpr (SECOND) {
                const uint32_t rc = rcode[slot][n];
                z[0] = __builtin_fma(code_value_d<MK, 0>(rc), rq, z[0]);
                z[1] = __builtin_fma(code_value_d<MK, 1>(rc), rq, z[1]);
                z[2] = __builtin_fma(code_value_d<MK, 2>(rc), rq, z[2]);
                z[3] = __builtin_fma(code_value_d<MK, 3>(rc), rq, z[3]);
              }
              *reinterpret_cast<uint32_t*>(smem + addr) = pack_codes_d<MK>(z[0], z[1], z[2], z[3], hi);
            }
          }
        });
        };
        constexpr bool MOVED = MOVE && !POOL;   // this layer moves tile (4, n)'s epilogue
        if constexpr (MOVED) {
          uint32_t* xa = reinterpret_cast<uint32_t*>(smem + C::OFF_Q4);   // [tile][16 values][64 lanes]
          if constexpr (XN >= 0) {
#pragma unroll
            for (int v = 0; v < 16; ++v) xa[(XN * 16 + v) * 64 + lane] = (uint32_t)c[MBW][XN][v];
            wave_lds_sync();
            epi_runs(std::integral_constant<int, 0>{}, std::integral_constant<int, MBW * 4>{});
          } else {
            epi_runs(std::integral_constant<int, 0>{}, std::integral_constant<int, MBW * 4>{});
            wave_lds_sync();
#pragma unroll
            for (int v = 0; v < 16; ++v) c[MBW][MV][v] = (int)xa[(MV * 16 + v) * 64 + lane];
            epi_runs(std::integral_constant<int, MBW * 4>{}, std::integral_constant<int, MBW * 4 + 4>{});
          }
        } else {
          epi_runs(std::integral_constant<int, 0>{}, std::integral_constant<int, NAF * 4>{});
        }
        if (has_next) store_consts((n_conv + 1) & 1, kn);
        __syncthreads();
      };

      for (int blk = 0; blk < p.blocks; ++blk) {
        const bool pool = p.pool_every > 0 && blk % p.pool_every == p.pool_every - 1;
        if (pool) conv(std::false_type{}, std::true_type{}, std::integral_constant<int, 0>{}, 2 * blk);
        else conv(std::false_type{}, std::false_type{}, std::integral_constant<int, 0>{}, 2 * blk);
        conv(std::true_type{}, std::false_type{}, std::integral_constant<int, C::S % NBUF>{}, 2 * blk + 1);
      }
    }

    // ---- heads input (bf16 networks): the low part h - bf16(h) of the fp32
    // residual as bf16 rows [square][F] at OFF_X, H holding bf16(h); int8
    // networks read the final codes from H and convert them in registers
    if constexpr (!QUANT) {
      using RX = Rot<C::RBX>;
#pragma unroll
      for (int m = 0; m < NAF; ++m)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int ch0 = blk_of(m) * 32 + 8 * q + 4 * lhi;
#pragma unroll
          for (int n = n_lo(m); n < n_hi(m); ++n) {
            const int j = n * 32 + l32;
            *reinterpret_cast<uint2*>(smem + C::OFF_X + j * C::RBX + (RX::pos(ch0 >> 3, RX::sw(j)) << 4) + 8 * lhi) =
                make_uint2(rlo[m][n][2 * q], rlo[m][n][2 * q + 1]);
          }
        }
    }
  };
  if (wave == 0) trunk(std::integral_constant<int, 0>{}, std::integral_constant<int, -1>{});
  else if (wave == 1) trunk(std::integral_constant<int, 1>{}, std::integral_constant<int, -1>{});
  else if (wave == 2) trunk(std::integral_constant<int, -1>{}, std::integral_constant<int, MOVE ? 0 : -1>{});
  else trunk(std::integral_constant<int, -1>{}, std::integral_constant<int, MOVE ? 1 : -1>{});
  __syncthreads();
  // ---- heads, shared by the four waves
  dep_heads4<MK>(p, smem, legal, policy, value, wdl, b, wave, lane);
}


}  // namespace
