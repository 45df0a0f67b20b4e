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
// The K loop runs over the nine taps; each tap's K steps are unrolled with
// compile-time register indices, so accumulators stay in the accumulation
// registers, weight fragments are double-buffered one prefetch group ahead
// (crossing taps and layers), and the LDS fragments of step k+1 are read while
// the MFMAs of step k run.  The epilogue (bias, residual, activation,
// requantisation) runs once per layer, followed by one workgroup barrier; its
// per-channel constants are staged through LDS one layer ahead.
//
// Activation layout in LDS: [board][square][channel], one row of F channels
// per square, stored in 16-byte chunks whose position is XOR-swizzled by the
// square index so that the 16 lanes of a ds_read_b128 group (16 consecutive
// squares, same logical chunk) hit 16 different bank groups.
//
// bf16 networks keep the residual stream (every block input h) in fp32 in the
// registers of the wave that produces it: each wave owns the same output tile
// in every layer, so the residual of an output element lives in the lane that
// computes it.  LDS holds bf16(h), the convolution operand.  The heads read h
// as bf16(h) + bf16(h - bf16(h)).
//
// MFMA output layout (32x32 blocks): lane l holds column l%32 and rows
// 8*(v/4) + 4*(l/32) + v%4 of its 16 accumulators v, i.e. four runs of four
// consecutive channels of one square, which the epilogue packs and stores with
// one LDS write per run.
#include "az_internal.h"
#include "az_mfma_common.h"

#include <math.h>

#include <type_traits>

namespace {

// LDS row address and swizzle of lane square j of half-board block nb for a tap.
// A tap outside the board reads the all-zero region instead, at the bank slot
// its (virtual) square r*8 + c would occupy: the slots a shifted window leaves
// free, so the 16 lanes of a read group never collide.
template <int RB_IN>
__device__ __forceinline__ void tap_row(int tap, int in_off, int zero_off, int nb, int l32, int& row,
                                        int& sw) {
  const int dy = tap / 3 - 1, dx = tap % 3 - 1;
  const int bl = nb >> 1, j = ((nb & 1) << 5) + l32;
  const int r = (j >> 3) + dy, c = (j & 7) + dx;
  const bool ok = (unsigned)r < 8u && (unsigned)c < 8u;
  const int src = r * 8 + c;
  const int ra = in_off + (bl * 64 + src) * RB_IN, rz = zero_off + ((src * RB_IN) & 255);
  const int msk = -(int)ok;  // branch-free select keeps the tap loop one basic block
  row = (ra & msk) | (rz & ~msk);
  sw = swz<RB_IN>(src);
}

// Tile shape: the wave owns MBW 32-channel blocks x NBW 32-square blocks; the
// workgroup is WM x WN waves; G consecutive K steps form one weight prefetch
// group; OCC workgroups share a compute unit.
template <int MK, int F, int MBW, int NBW, int WM, int WN, int G, int OCC, int NBUF_>
struct Cfg {
  using T = Mk<MK>;
  static constexpr int NW = WM * WN, NT = 64 * NW;
  static constexpr int BPW = NBW * WN / 2;  // boards per workgroup
  static constexpr int NMB = F / 32;
  static_assert(NMB == MBW * WM, "channel tiling");
  static_assert(NBW % 2 == 0, "board tiling");
  static constexpr int RB = F * T::ES;  // bytes per square row, tower tensors
  static constexpr int BUF = BPW * 64 * RB;
  static constexpr int OFF_H = 0, OFF_T = BUF, OFF_Z = 2 * BUF;
  static constexpr int ZB = cmax(RB, 256);  // zero region: a 256-byte bank window at least
  static constexpr int RBX = 2 * F;  // bf16 row bytes of the heads' input
  static constexpr int OFF_X = OFF_T;
  static constexpr int LBMAX = (AZ_MAX_POLICY + 1) * 64;  // floats per board, logits + u
  // per-layer epilogue constants, double-buffered: [2 slots][bias F] floats, or
  // for quantised nets [2 slots][qbias F | qmul F] doubles
  static constexpr int OFF_K = 2 * BUF + ZB;
  static constexpr int KSLOT = MK == MK_BF16 ? 4 * F : 16 * F;
  // head row constants (scale, bias) and the softmax / value reductions sit past
  // every other region: they are written at the start and read at the end
  static constexpr int OFF_HC = (cmax(cmax(OFF_K + 2 * KSLOT, OFF_X + BPW * 64 * RBX), BPW * LBMAX * 4) + 15) & ~15;
  static constexpr int RED_PER_BOARD = 32;  // floats: [0,8) sum groups, [8,12) max per wave, [16,24) value groups
  static constexpr int OFF_RED = OFF_HC + 2 * AZ_HEAD_ROWS * 4;
  static constexpr int SMEM = OFF_RED + BPW * RED_PER_BOARD * 4;
  static_assert(SMEM * OCC <= 160 * 1024, "LDS");
  static_assert(NW % BPW == 0, "every board gets a whole number of waves at the end");
  static constexpr int CPT = F / T::KS;  // K steps per tap
  static_assert(CPT % G == 0, "group size");
  static constexpr int S = 9 * CPT;      // K steps per layer
  static constexpr int GPL = S / G;      // prefetch groups per layer
  static constexpr int NBUF = NBUF_;     // weight prefetch ring depth (groups)
  static_assert((2 * GPL) % NBUF == 0, "every block's first conv starts at ring slot 0");
  static constexpr int STEP_BYTES = NMB * 64 * T::FB;
  static constexpr size_t LAYER_BYTES = (size_t)S * STEP_BYTES;
  static constexpr int NBH = (2 * BPW + NW - 1) / NW;  // head N-blocks per wave
};

template <int MK, int F, int MBW, int NBW, int WM, int WN, int G, int OCC, int NBUF_, int IL>
__global__ __attribute__((amdgpu_flat_work_group_size(64 * WM * WN, 64 * WM * WN),
                          amdgpu_waves_per_eu(OCC, OCC))) void
az_net_kernel(AzDevNet p, const float* __restrict__ planes, const uint8_t* __restrict__ legal, int B,
              float* __restrict__ policy, float* __restrict__ value) {
  using C = Cfg<MK, F, MBW, NBW, WM, WN, G, OCC, NBUF_>;
  using T = typename C::T;
  using SB = Mk<MK_BF16>;
  using frag_t = typename T::frag;
  using acc_t = typename T::acc;
  constexpr bool QUANT = MK != MK_BF16;
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

  // fp32 residual stream of the wave's output tile (bf16 networks)
  float res[QUANT ? 1 : MBW][QUANT ? 1 : NBW][16];

  // The four-board tilings (one workgroup per CU) have registers to spare
  // outside the tower: they load the stem's and the heads' weights early.
  constexpr bool ROOMY = OCC == 1 && NBW >= 4;
  // Stem weights (bf16, K = 288 in nine taps of two steps): a ring of SR taps,
  // the first SR - 1 loaded here, ahead of the input planes, so that their
  // latency overlaps the ingest: all nine taps, or double-buffered.
  constexpr int SR = ROOMY ? 9 : 2, SSTEP = NMB * 64 * 16;
  const uint8_t* sw8 = static_cast<const uint8_t*>(p.stem_w) + (size_t)(mb0 * 64 + lane) * 16;
  SB::frag sa[SR][2][MBW];
  auto load_stem_tap = [&](int tap, SB::frag(&dst)[2][MBW]) {
#pragma unroll
    for (int s = 0; s < 2; ++s)
#pragma unroll
      for (int m = 0; m < MBW; ++m) dst[s][m] = g_frag<MK_BF16>(sw8 + (tap * 2 + s) * SSTEP + m * 64 * 16);
  };
  static_for<0, SR - 1>([&](auto t_c) { load_stem_tap(decltype(t_c)::value, sa[decltype(t_c)::value]); });

  // ---- ingest: zero row, planes -> bf16 [board][square][32 channels] at OFF_T
  for (int i = tid; i < C::ZB / 16; i += NT)
    *reinterpret_cast<i32x4*>(smem + OFF_Z + i * 16) = i32x4{0, 0, 0, 0};
  // One item = 8 input planes of one board: lane = square, eight plane loads (each
  // coalesced over the wave), one 16-byte LDS store.  Items are wave-uniform and
  // every load is issued before the first is used.
  {
    constexpr int ITEMS = BPW * 4, PER = (ITEMS + NW - 1) / NW;
    float pv[PER][8];
#pragma unroll
    for (int it = 0; it < PER; ++it) {
      const int item = w + it * NW, bl = item >> 2, k = item & 3, b = b0 + bl;
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        // unconditional load (clamped to plane 0 of board 0) so that no branch
        // separates a load from the next one
        const int c = 8 * k + t;
        const bool ok = item < ITEMS && b < B && c < Cin;
        const float x = planes[ok ? ((size_t)b * Cin + c) * 64 + lane : (size_t)lane];
        pv[it][t] = ok ? x : 0.0f;
      }
    }
#pragma unroll
    for (int it = 0; it < PER; ++it) {
      const int item = w + it * NW, bl = item >> 2, k = item & 3;
      if (item < ITEMS)
        *reinterpret_cast<uint4*>(smem + OFF_T + (bl * 64 + lane) * 64 + ((k ^ swz<64>(lane)) << 4)) =
            make_uint4(pack_bf16x2(pv[it][0], pv[it][1]), pack_bf16x2(pv[it][2], pv[it][3]),
                       pack_bf16x2(pv[it][4], pv[it][5]), pack_bf16x2(pv[it][6], pv[it][7]));
    }
  }

  // first weight group of the tower, in flight during the stem
  // Weight fragments: a ring of NBUF prefetch groups; group g of a layer lives in
  // buffer g % NBUF and is loaded NBUF - 1 groups before its use.
  // The stream is read through a buffer resource: the lane's offset is a
  // constant VGPR and a group's byte offset a scalar, so weight loads cost no
  // vector address arithmetic in the K loop.
  constexpr int NBUF = C::NBUF;
  const __amdgpu_buffer_rsrc_t twr = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<void*>(p.tower_w), (short)0, (int)(2 * p.blocks * C::LAYER_BYTES), 0x00020000);
  const int tvoff = (mb0 * 64 + lane) * T::FB;
  frag_t A[NBUF][G][MBW];
  auto load_group = [&](frag_t(&dst)[G][MBW], int soff) {
#pragma unroll
    for (int s = 0; s < G; ++s)
#pragma unroll
      for (int m = 0; m < MBW; ++m) {
        const int o = soff + s * C::STEP_BYTES + m * 64 * T::FB;
        if constexpr (T::FB == 16) {
          dst[s][m] = __builtin_bit_cast(frag_t, __builtin_amdgcn_raw_buffer_load_b128(twr, tvoff, o, 0));
        } else {
          const i32x4 lo = __builtin_amdgcn_raw_buffer_load_b128(twr, tvoff, o, 0);
          const i32x4 hi = __builtin_amdgcn_raw_buffer_load_b128(twr, tvoff, o + 16, 0);
          dst[s][m] = __builtin_bit_cast(frag_t, i32x8{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]});
        }
      }
  };
  static_for<0, NBUF - 1>([&](auto i_c) {
    constexpr int i = decltype(i_c)::value;
    load_group(A[i], i * G * C::STEP_BYTES);
  });
  // per-layer epilogue constants: thread t < KSLOT/16 carries 16-byte chunk t of
  // the slot ([bias] floats, or [qbias | qmul] doubles)
  constexpr int KCH = C::KSLOT / 16;
  auto load_consts = [&](int k) -> float4 {  // k = 1 + conv index (0 = stem)
    if (tid >= KCH) return make_float4(0.f, 0.f, 0.f, 0.f);
    if constexpr (QUANT) {
      const double* src = tid < F / 2 ? p.qbias + (size_t)k * F + 2 * tid : p.qmul + (size_t)k * F + 2 * (tid - F / 2);
      return *reinterpret_cast<const float4*>(src);
    } else {
      return *reinterpret_cast<const float4*>(p.bias + (size_t)k * F + tid * 4);
    }
  };
  auto store_consts = [&](int slot, const float4& v) {
    if (tid < KCH) *reinterpret_cast<float4*>(smem + C::OFF_K + slot * C::KSLOT + tid * 16) = v;
  };
  static_assert(NT >= KCH, "constant staging needs a thread per 16-byte chunk");
  store_consts(0, load_consts(1));
  if (tid < AZ_HEAD_ROWS / 2)  // [scale 96 | bias 96] floats
    *reinterpret_cast<float4*>(smem + C::OFF_HC + tid * 16) =
        *reinterpret_cast<const float4*>(tid < AZ_HEAD_ROWS / 4 ? p.head_sc + tid * 4 : p.head_bc + (tid - AZ_HEAD_ROWS / 4) * 4);
  static_assert(NT >= AZ_HEAD_ROWS / 2, "head constant staging");
  __syncthreads();

  // ---- stem: bf16 3x3 conv over 32 (padded) input channels, K = 288
  {
    f32x16 sacc[MBW][NBW];
    int row[NBW], sw[NBW], nrow[NBW], nsw[NBW];
    SB::frag bc[NBW], bn[NBW];
#pragma unroll
    for (int n = 0; n < NBW; ++n) {
      tap_row<64>(0, OFF_T, OFF_Z, nb0 + n, l32, row[n], sw[n]);
      bc[n] = lds_frag<MK_BF16>(smem, row[n], sw[n], lhi);
    }
#pragma unroll
    for (int tap = 0; tap < 9; ++tap) {
      if (tap + SR - 1 < 9) load_stem_tap(tap + SR - 1, sa[(tap + SR - 1) % SR]);
      if (tap + 1 < 9) {
#pragma unroll
        for (int n = 0; n < NBW; ++n) tap_row<64>(tap + 1, OFF_T, OFF_Z, nb0 + n, l32, nrow[n], nsw[n]);
      }
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        if (s == 0) {
#pragma unroll
          for (int n = 0; n < NBW; ++n) bn[n] = lds_frag<MK_BF16>(smem, row[n], sw[n], 2 + lhi);
        } else if (tap + 1 < 9) {
#pragma unroll
          for (int n = 0; n < NBW; ++n) bn[n] = lds_frag<MK_BF16>(smem, nrow[n], nsw[n], lhi);
        }
#pragma unroll
        for (int m = 0; m < MBW; ++m)
#pragma unroll
          for (int n = 0; n < NBW; ++n)
            sacc[m][n] = SB::mma(sa[tap % SR][s][m], bc[n], (tap == 0 && s == 0) ? f32x16{} : sacc[m][n]);
#pragma unroll
        for (int n = 0; n < NBW; ++n) bc[n] = bn[n];
      }
      if (tap + 1 < 9) {
#pragma unroll
        for (int n = 0; n < NBW; ++n) {
          row[n] = nrow[n];
          sw[n] = nsw[n];
        }
      }
    }
    // epilogue: bias, activation, store in the tower format at OFF_H
#pragma unroll
    for (int m = 0; m < MBW; ++m)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int ch0 = (mb0 + m) * 32 + 8 * q + 4 * lhi;
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
          const int nb = nb0 + n, bl = nb >> 1, j = ((nb & 1) << 5) + l32;
          const f32x16& v = sacc[m][n];
          const int rowo = OFF_H + (bl * 64 + j) * RB;
          if constexpr (!QUANT) {
            const float y0 = act_fn(v[4 * q + 0] + bb.x, cap), y1 = act_fn(v[4 * q + 1] + bb.y, cap);
            const float y2 = act_fn(v[4 * q + 2] + bb.z, cap), y3 = act_fn(v[4 * q + 3] + bb.w, cap);
            res[m][n][4 * q + 0] = y0;
            res[m][n][4 * q + 1] = y1;
            res[m][n][4 * q + 2] = y2;
            res[m][n][4 * q + 3] = y3;
            *reinterpret_cast<uint2*>(smem + rowo + (((ch0 >> 3) ^ swz<RB>(j)) << 4) + 8 * lhi) =
                make_uint2(pack_bf16x2(y0, y1), pack_bf16x2(y2, y3));
          } else {
            // the stem's sum comes from the bf16 matrix instruction in fp32; the
            // rescale and rounding of its code are taken in float64
            const float hi = p.qhi[0];
            *reinterpret_cast<uint32_t*>(smem + rowo + (((ch0 >> 4) ^ swz<RB>(j)) << 4) + (ch0 & 15)) =
                pack_codes_d<MK>(__builtin_fma((double)v[4 * q + 0], mq[0], bq[0]),
                                 __builtin_fma((double)v[4 * q + 1], mq[1], bq[1]),
                                 __builtin_fma((double)v[4 * q + 2], mq[2], bq[2]),
                                 __builtin_fma((double)v[4 * q + 3], mq[3], bq[3]), hi);
          }
        }
      }
  }
  __syncthreads();

  // ---- residual tower: per block conv1 (H -> T) and conv2 (T -> H, + residual)
  {
    constexpr int CPT = C::CPT, GPL = C::GPL, GPT = CPT / G;
    acc_t c[MBW][NBW];
    const int nconv = 2 * p.blocks;

    auto conv = [&](auto second_c, auto lb_c, int n_conv) {
      constexpr bool SECOND = decltype(second_c)::value;
      constexpr int LB = decltype(lb_c)::value;  // ring slot of the layer's first group
      const int wl = n_conv * (int)C::LAYER_BYTES;  // byte offset of the layer in the stream
      const bool has_next = n_conv + 1 < nconv;
      const int in_off = SECOND ? OFF_T : OFF_H;
      const int out_off = SECOND ? OFF_H : OFF_T;
      // the next layer's epilogue constants, parked in LDS before this layer's barrier
      const float4 kn = has_next ? load_consts(n_conv + 2) : make_float4(0.f, 0.f, 0.f, 0.f);
      const float* kslot = reinterpret_cast<const float*>(smem + C::OFF_K + (n_conv & 1) * C::KSLOT);
      // B fragments of one K step: rows of the current tap, chunk of channel step cs
      int row[NBW], sw[NBW], nrow[NBW], nsw[NBW];
      auto rows_for = [&](int tap, int(&rr)[NBW], int(&ss)[NBW]) {
#pragma unroll
        for (int n = 0; n < NBW; ++n) tap_row<RB>(tap, in_off, OFF_Z, nb0 + n, l32, rr[n], ss[n]);
      };
      auto load_b = [&](const int(&rr)[NBW], const int(&ss)[NBW], int cs, frag_t(&dst)[NBW]) {
        const int lc = MK == MK_F8 ? 4 * cs + 2 * lhi : 2 * cs + lhi;
#pragma unroll
        for (int n = 0; n < NBW; ++n) dst[n] = lds_frag<MK>(smem, rr[n], ss[n], lc);
      };
      frag_t bc[NBW], bn[NBW];
      rows_for(0, row, sw);
      load_b(row, sw, 0, bc);

      // One tap: CPT K steps in GPT prefetch groups; R0 = ring slot of its first
      // group.  The first step of the layer starts its accumulators from zero.
      auto tap_body = [&](auto r0_c, auto first_c, int tap) {
        constexpr int R0 = decltype(r0_c)::value;
        constexpr bool FIRST = decltype(first_c)::value;
        // Branch-free body: prefetches past the network's last layer re-read this
        // layer (never used); after the last tap the next tap's rows and fragments
        // point inside the board or at the zero region.
        rows_for(tap + 1, nrow, nsw);
        static_for<0, CPT>([&](auto cs_c) {
          constexpr int cs = decltype(cs_c)::value;
          constexpr int gs = cs / G, sg = cs % G;
          constexpr int cur = (R0 + gs) % NBUF;
          auto& Acur = A[cur];
          if constexpr (sg == 0) {
            // group tap*GPT + gs + NBUF-1 of this layer, i.e. of the next layer past
            // the end (layers are contiguous)
            const int gi = tap * GPT + gs + NBUF - 1;
            load_group(A[(cur + NBUF - 1) % NBUF], wl + ((has_next || gi < GPL) ? gi * G * C::STEP_BYTES : 0));
          }
          if constexpr (cs + 1 < CPT) load_b(row, sw, cs + 1, bn);
          else load_b(nrow, nsw, 0, bn);
#pragma unroll
          for (int m = 0; m < MBW; ++m)
#pragma unroll
            for (int n = 0; n < NBW; ++n)
              c[m][n] = T::mma(Acur[sg][m], bc[n], (FIRST && cs == 0) ? acc_t{} : c[m][n]);
#pragma unroll
          for (int n = 0; n < NBW; ++n) bc[n] = bn[n];
          if constexpr (IL) {
            // interleave: each MFMA is followed by one of the next step's LDS
            // reads, then by one of the prefetch group's weight loads
            constexpr int PER = MK == MK_F8 ? 2 : 1;  // instructions per fragment
            constexpr int NDS = NBW * PER, NVM = sg == 0 ? G * MBW * PER : 0, NMF = MBW * NBW;
            static_for<0, NMF>([&](auto i_c) {
              constexpr int i = decltype(i_c)::value;
              __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
              if constexpr (i < NDS) __builtin_amdgcn_sched_group_barrier(0x100, i + 1 == NMF ? NDS - i : 1, 0);
              if constexpr (i < NVM) __builtin_amdgcn_sched_group_barrier(0x020, i + 1 == NMF ? NVM - i : 1, 0);
            });
          }
        });
#pragma unroll
        for (int n = 0; n < NBW; ++n) {
          row[n] = nrow[n];
          sw[n] = nsw[n];
        }
      };
      // taps 1..8 in a runtime loop unrolled by U taps, U the period of the ring
      // slot of a tap's first group; the remainder is peeled
      constexpr int U = NBUF / gcd_c(GPT, NBUF), NIT = 8 / U, REM = 8 % U;
      tap_body(std::integral_constant<int, LB>{}, std::true_type{}, 0);
#pragma nounroll
      for (int it = 0; it < NIT; ++it) {
        static_for<0, U>([&](auto u_c) {
          constexpr int u = decltype(u_c)::value;
          tap_body(std::integral_constant<int, (LB + (1 + u) * GPT) % NBUF>{}, std::false_type{},
                   1 + it * U + u);
        });
      }
      static_for<0, REM>([&](auto u_c) {
        constexpr int u = decltype(u_c)::value, t = 1 + NIT * U + u;
        tap_body(std::integral_constant<int, (LB + t * GPT) % NBUF>{}, std::false_type{}, t);
      });

      // epilogue
      float hi = 0.0f;
      double rq = 0.0;
      if constexpr (QUANT) {
        hi = p.qhi[n_conv + 1];
        rq = SECOND ? p.qres[n_conv + 1] : 0.0;
      }
      // The epilogue walks the wave's rows in runs k = (m, q) of 4 channels.  Its
      // LDS reads (the run's per-channel constants and, for the second conv of
      // a quantised block, the residual codes, read in place before this lane
      // overwrites them) are issued EP_AHEAD runs ahead of their arithmetic, in
      // a ring of EP_AHEAD + 1 slots, so that no read latency is exposed (two
      // runs in the four-board tiling, one in the two-board one; the one-board
      // tiling has no registers to spare for the float64 constants and reads
      // them in place).  Quantised layers requantise in float64: z = acc * qmul
      // + qbias (+ residual code * qres), rounded to the code grid and clamped.
      constexpr int NRUN = MBW * 4, EP_AHEAD = QUANT ? (NBW >= 4 ? 2 : (BPW == 1 ? 0 : 1)) : 0, EP_RING = EP_AHEAD + 1;
      constexpr bool RCODE = QUANT && SECOND;
      struct KQ { double b[4], m[4]; };
      float4 kb[QUANT ? 1 : EP_RING];
      KQ kq[QUANT ? EP_RING : 1];
      uint32_t rcode[RCODE ? EP_RING : 1][RCODE ? NBW : 1];
      auto ep_addr = [&](int m, int q, int n) {
        const int nb = nb0 + n, bl = nb >> 1, j = ((nb & 1) << 5) + l32;
        const int ch0 = (mb0 + m) * 32 + 8 * q + 4 * lhi;
        const int rowo = out_off + (bl * 64 + j) * RB;
        if constexpr (QUANT) return rowo + (((ch0 >> 4) ^ swz<RB>(j)) << 4) + (ch0 & 15);
        else return rowo + (((ch0 >> 3) ^ swz<RB>(j)) << 4) + 8 * lhi;
      };
      auto ep_load = [&](auto k_c) {
        constexpr int k = decltype(k_c)::value, m = k / 4, q = k % 4, slot = k % EP_RING;
        const int ch0 = (mb0 + m) * 32 + 8 * q + 4 * lhi;
        if constexpr (QUANT) {
          const double* kd = reinterpret_cast<const double*>(kslot);
#pragma unroll
          for (int r = 0; r < 4; r += 2) {
            const double2 b2 = *reinterpret_cast<const double2*>(kd + ch0 + r);
            const double2 m2 = *reinterpret_cast<const double2*>(kd + F + ch0 + r);
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
              y0 = act_fn(y0 + res[m][n][4 * q + 0], cap);
              y1 = act_fn(y1 + res[m][n][4 * q + 1], cap);
              y2 = act_fn(y2 + res[m][n][4 * q + 2], cap);
              y3 = act_fn(y3 + res[m][n][4 * q + 3], cap);
              res[m][n][4 * q + 0] = y0;
              res[m][n][4 * q + 1] = y1;
              res[m][n][4 * q + 2] = y2;
              res[m][n][4 * q + 3] = y3;
            } else {
              y0 = act_fn(y0, cap);
              y1 = act_fn(y1, cap);
              y2 = act_fn(y2, cap);
              y3 = act_fn(y3, cap);
            }
            *reinterpret_cast<uint2*>(smem + addr) = make_uint2(pack_bf16x2(y0, y1), pack_bf16x2(y2, y3));
          } else {
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
      conv(std::false_type{}, std::integral_constant<int, 0>{}, 2 * blk);
      conv(std::true_type{}, std::integral_constant<int, GPL % NBUF>{}, 2 * blk + 1);
    }
  }

  // ---- heads: 1x1 convs F -> (P policy planes + 1 value row) as one bf16 GEMM
  const int P = p.policy_planes;
  const int NMV = P * 64;
  // Softmax and value: WPB waves per board.  The board's cells form groups g of
  // 1024; in group g lane l owns the four runs of 4 cells at g*1024 + u*256 + 4l
  // (u = 0..3), so that a wave's LDS reads, mask loads and policy stores are
  // contiguous.  Wave part p of the board takes groups p, p + WPB, ...  Its
  // legal mask is loaded here, in flight during the heads.
  constexpr int WPB = NW / BPW;
  constexpr int NGRP = (AZ_MAX_POLICY * 64 + 1023) / 1024;  // cell groups
  constexpr int NGW = (NGRP + WPB - 1) / WPB;               // groups per wave
  const int sbl = w / WPB, spart = w % WPB;
  const int sb = b0 + sbl;
  const bool svalid = sb < B;
  uint32_t mk0[NGW][4];
#pragma unroll
  for (int ii = 0; ii < NGW; ++ii)
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int c = 1024 * (spart + WPB * ii) + 256 * u + 4 * lane;
      const bool ok = svalid && c < NMV;
      const uint32_t x = *reinterpret_cast<const uint32_t*>(legal + (ok ? (size_t)sb * NMV + c : (size_t)0));
      mk0[ii][u] = ok ? x : 0u;
    }
  {
    constexpr int HS = F / 16, RBX = C::RBX, OFF_X = C::OFF_X, NBH = C::NBH;
    // head weights: in flight during the conversion below where the registers
    // allow, else loaded after it
    SB::frag ha[HS][3];
    auto load_head_w = [&]() {
      const uint8_t* hw = static_cast<const uint8_t*>(p.head_w) + (size_t)lane * 16;
#pragma unroll
      for (int s = 0; s < HS; ++s)
#pragma unroll
        for (int m = 0; m < 3; ++m) ha[s][m] = g_frag<MK_BF16>(hw + ((s * 3 + m) * 64) * 16);
    };
    if constexpr (ROOMY) load_head_w();
    if constexpr (QUANT) {
      // codes -> exact bf16 values (int8 and e4m3 values are bf16-representable)
      for (int idx = tid; idx < BPW * 64 * (F / 8); idx += NT) {
        const int k = idx % (F / 8), sq = (idx / (F / 8)) & 63, bl = idx / (64 * (F / 8));
        const uint2 v = *reinterpret_cast<const uint2*>(
            smem + OFF_H + (bl * 64 + sq) * RB + (((k >> 1) ^ swz<RB>(sq)) << 4) + (k & 1) * 8);
        const uint4 o = make_uint4(pack_bf16x2(code_value<MK, 0>(v.x), code_value<MK, 1>(v.x)),
                                   pack_bf16x2(code_value<MK, 2>(v.x), code_value<MK, 3>(v.x)),
                                   pack_bf16x2(code_value<MK, 0>(v.y), code_value<MK, 1>(v.y)),
                                   pack_bf16x2(code_value<MK, 2>(v.y), code_value<MK, 3>(v.y)));
        *reinterpret_cast<uint4*>(smem + OFF_X + (bl * 64 + sq) * RBX + ((k ^ swz<RBX>(sq)) << 4)) = o;
      }
    } else {
      // low half of the fp32 residual: bf16(h - bf16(h)), same layout at OFF_X
#pragma unroll
      for (int m = 0; m < MBW; ++m)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int ch0 = (mb0 + m) * 32 + 8 * q + 4 * lhi;
#pragma unroll
          for (int n = 0; n < NBW; ++n) {
            const int nb = nb0 + n, bl = nb >> 1, j = ((nb & 1) << 5) + l32;
            float lo[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) lo[r] = res[m][n][4 * q + r] - bf16_round(res[m][n][4 * q + r]);
            *reinterpret_cast<uint2*>(smem + OFF_X + (bl * 64 + j) * RBX + (((ch0 >> 3) ^ swz<RBX>(j)) << 4) +
                                      8 * lhi) = make_uint2(pack_bf16x2(lo[0], lo[1]), pack_bf16x2(lo[2], lo[3]));
          }
        }
    }
    if constexpr (!ROOMY) load_head_w();
    __syncthreads();

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
        if constexpr (!QUANT) {
          const int rowh = OFF_H + (bl * 64 + j) * RBX;
#pragma unroll
          for (int s = 0; s < HS; ++s) {
            const SB::frag bfr = lds_frag<MK_BF16>(smem, rowh, swx, 2 * s + lhi);
#pragma unroll
            for (int m = 0; m < 3; ++m) hacc[k][m] = SB::mma(ha[s][m], bfr, hacc[k][m]);
          }
        }
      }
    }
    __syncthreads();
    // every row of every board: fma(acc, scale, bias) with the row constants
    // (policy rows leave pre-scaled by log2(e), rows past P are never read)
    float* L = reinterpret_cast<float*>(smem);
    const float* HC = reinterpret_cast<const float*>(smem + C::OFF_HC);
#pragma unroll
    for (int m = 0; m < 3; ++m)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int r0 = m * 32 + 8 * q + 4 * lhi;
        const float4 sc = *reinterpret_cast<const float4*>(HC + r0);
        const float4 bc = *reinterpret_cast<const float4*>(HC + AZ_HEAD_ROWS + r0);
#pragma unroll
        for (int k = 0; k < NBH; ++k) {
          const int nb = w + k * NW;
          if (nb < 2 * BPW) {
            const int bl = nb >> 1, j = ((nb & 1) << 5) + l32;
            float* dst = L + bl * C::LBMAX + r0 * 64 + j;
            dst[0] = __builtin_fmaf(hacc[k][m][4 * q + 0], sc.x, bc.x);
            dst[64] = __builtin_fmaf(hacc[k][m][4 * q + 1], sc.y, bc.y);
            dst[128] = __builtin_fmaf(hacc[k][m][4 * q + 2], sc.z, bc.z);
            dst[192] = __builtin_fmaf(hacc[k][m][4 * q + 3], sc.w, bc.w);
          }
        }
      }
  }
  __syncthreads();

  // ---- legal-move softmax and value head: WPB waves per board (board sbl, part spart)
  // Sums are taken in an order that does not depend on WPB, so every tiling
  // returns the same bits: each 64-chunk group (policy) or 64-unit group (value
  // hidden layer) is reduced across the lanes of one wave, and the group sums
  // are added in group order.
  {
    const float* L = reinterpret_cast<const float*>(smem);
    float* red = reinterpret_cast<float*>(smem + C::OFF_RED) + sbl * C::RED_PER_BOARD;
    const float* Lb = L + sbl * C::LBMAX;
    float* pol = policy + (size_t)sb * NMV;
    const int H = p.value_hidden;
    // logits are stored as z * log2(e): p_i = 2^(zl_i - max zl) / sum over legal cells.
    // Illegal cells carry -inf through the max and contribute exactly 0.
    float e[NGW][16];
    float mx = -INFINITY;
#pragma unroll
    for (int ii = 0; ii < NGW; ++ii)
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int c = 1024 * (spart + WPB * ii) + 256 * u + 4 * lane;
        const bool in = c < NMV;
        const float4 z4 = in ? *reinterpret_cast<const float4*>(Lb + c) : make_float4(0.f, 0.f, 0.f, 0.f);
        const float zz[4] = {z4.x, z4.y, z4.z, z4.w};
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          const bool ok = in && ((mk0[ii][u] >> (8 * t)) & 0xffu);
          e[ii][4 * u + t] = ok ? zz[t] : -INFINITY;
          mx = fmaxf(mx, e[ii][4 * u + t]);
        }
      }
    mx = wave_max(mx);
    if (lane == 0) red[8 + spart] = mx;
    __syncthreads();
    float bmx = red[8];
#pragma unroll
    for (int t = 1; t < WPB; ++t) bmx = fmaxf(bmx, red[8 + t]);
    const float msub = bmx == -INFINITY ? 0.0f : bmx;
#pragma unroll
    for (int ii = 0; ii < NGW; ++ii) {
      float gsum = 0.0f;
#pragma unroll
      for (int t = 0; t < 16; ++t) {
        e[ii][t] = __builtin_amdgcn_exp2f(e[ii][t] - msub);  // exp2(-inf) = 0
        gsum += e[ii][t];
      }
      gsum = wave_sum(gsum);
      if (lane == 0 && spart + WPB * ii < NGRP) red[spart + WPB * ii] = gsum;
    }
    // value head inputs and hidden-unit groups r (unit 64 r + lane) of this wave
    float u[64];
#pragma unroll
    for (int s4 = 0; s4 < 64; s4 += 4) {
      const float4 t4 = *reinterpret_cast<const float4*>(Lb + NMV + s4);
      u[s4] = t4.x;
      u[s4 + 1] = t4.y;
      u[s4 + 2] = t4.z;
      u[s4 + 3] = t4.w;
    }
    if (p.value_conv_relu) {
#pragma unroll
      for (int s4 = 0; s4 < 64; ++s4) u[s4] = fmaxf(u[s4], 0.0f);
    }
    const int ngv = (H + 63) >> 6;  // hidden-unit groups (H <= 512: at most 8)
    for (int r = spart; r < ngv; r += WPB) {
      const int k = 64 * r + lane;
      const bool ok = k < H;
      const float4* src = reinterpret_cast<const float4*>(p.fc1_t) + (ok ? k : 0);
      float4 wr[16];
#pragma unroll
      for (int s4 = 0; s4 < 16; ++s4) wr[s4] = src[(size_t)s4 * H];
      const float gb = p.fc1_b[ok ? k : 0], w2r = p.fc2_w[ok ? k : 0];
      float g = ok ? gb : 0.0f;
      const float w2 = ok ? w2r : 0.0f;
#pragma unroll
      for (int s4 = 0; s4 < 16; ++s4)
        g += wr[s4].x * u[4 * s4] + wr[s4].y * u[4 * s4 + 1] + wr[s4].z * u[4 * s4 + 2] + wr[s4].w * u[4 * s4 + 3];
      const float vsum = wave_sum(w2 * fmaxf(g, 0.0f));
      if (lane == 0) red[16 + r] = vsum;
    }
    __syncthreads();
    float tot = 0.0f;
#pragma unroll
    for (int g = 0; g < NGRP; ++g) tot += (1024 * g < NMV) ? red[g] : 0.0f;
    const float inv = tot > 0.0f ? 1.0f / tot : 0.0f;
    if (svalid) {
#pragma unroll
      for (int ii = 0; ii < NGW; ++ii)
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int c = 1024 * (spart + WPB * ii) + 256 * u + 4 * lane;
          if (c < NMV)
            *reinterpret_cast<float4*>(pol + c) =
                make_float4(e[ii][4 * u] * inv, e[ii][4 * u + 1] * inv, e[ii][4 * u + 2] * inv, e[ii][4 * u + 3] * inv);
        }
      if (spart == 0 && lane == 0) {
        float vs = 0.0f;
        for (int r = 0; r < ngv; ++r) vs += red[16 + r];
        value[sb] = tanhf(vs + p.fc2_b);
      }
    }
  }
}

template <int MK, int F, int MBW, int NBW, int WM, int WN, int G, int OCC, int NBUF, int IL>
hipError_t launch_cfg(const AzDevNet& n, const float* planes, const uint8_t* legal, int B,
                      float* policy, float* value, hipStream_t s) {
  using C = Cfg<MK, F, MBW, NBW, WM, WN, G, OCC, NBUF>;
  const int grid = (B + C::BPW - 1) / C::BPW;
  hipLaunchKernelGGL((az_net_kernel<MK, F, MBW, NBW, WM, WN, G, OCC, NBUF, IL>), dim3(grid), dim3(C::NT), 0, s,
                     n, planes, legal, B, policy, value);
  return hipGetLastError();
}

// K-loop weight stream per tiling: G-step prefetch groups, a ring of NB groups
// (loaded NB-1 groups ahead), IL = explicit MFMA / LDS / load interleave.
// Deepest ring of at most `want` groups that tiles two layers of `gpl` groups.
constexpr int ring_depth(int want, int gpl) {
  return want <= 2 ? 2 : ((2 * gpl) % want == 0 ? want : ring_depth(want - 1, gpl));
}

template <int MK, int F>
struct Sched {
  static constexpr int CPT = F / Mk<MK>::KS;
  static constexpr bool BF = MK == MK_BF16, I8 = MK == MK_I8;
  // Multi-board tilings: int8 streams one step per group with a ring of 12 in
  // the large tiling (F <= 128) and 8 in the medium one (whose two workgroups per
  // compute unit leave no registers for more), fp8 (32-byte fragments) a ring
  // of 6 in the large tiling and 4 in the medium one, bf16 two-step groups with
  // a ring of 3 in the large tiling up to F = 128 (768 boards: 461 us against 486
  // for a ring of 2; 1,024 boards unchanged) and of 2 elsewhere (its fp32
  // residual stream needs the registers).
  static constexpr int GL = BF ? 2 : 1, NL = BF ? (F <= 128 ? 3 : 2) : (I8 ? (F <= 128 ? 12 : 8) : 6), IL_L = 1;
  static constexpr int GM = GL, NM = BF ? 2 : (I8 ? 8 : 4), IL_M = 1;
  // small (one board per workgroup): one-step groups; a wave's K step is two
  // MFMAs, so covering a load from the Infinity Cache takes a deep ring: 18
  // steps for int8, 12 for bf16 (measured best; 16 and 18 are slower or
  // spill), 8 for fp8 (32-byte fragments); bf16 at F = 256 two-step groups with
  // a ring of 2 (the bf16 residual stream needs the registers)
  static constexpr bool W256 = BF && F == 256;
  static constexpr int GS = W256 ? 2 : 1, NS = W256 ? 2 : (I8 ? 18 : (BF ? 12 : 8)), IL_S = 1;
};

// Tilings (wave tile = MBW*32 channels x NBW half-boards):
//   1 large:  4 boards per workgroup (2 for F = 256), 64 ch x 2 boards per wave
//   2 small:  1 board per workgroup
//   3 medium: 2 boards per workgroup, two workgroups per compute unit (F = 64, 128)
template <int MK, int F>
hipError_t launch_f(int tiling, const AzDevNet& n, const float* planes, const uint8_t* legal, int B,
                    float* policy, float* value, hipStream_t s) {
  using S = Sched<MK, F>;
  if constexpr (F == 128) {
    if (tiling == 1)
      return launch_cfg<MK, 128, 2, 4, 2, 2, S::GL, 1, ring_depth(S::NL, 9 * S::CPT / S::GL), S::IL_L>(n, planes, legal, B, policy, value, s);
    if (tiling == 3)
      return launch_cfg<MK, 128, 2, 2, 2, 2, S::GM, 2, ring_depth(S::NM, 9 * S::CPT / S::GM), S::IL_M>(n, planes, legal, B, policy, value, s);
    return launch_cfg<MK, 128, 1, 2, 4, 1, S::GS, 2, ring_depth(S::NS, 9 * S::CPT / S::GS), S::IL_S>(n, planes, legal, B, policy, value, s);
  } else if constexpr (F == 256) {
    if (tiling == 1)
      return launch_cfg<MK, 256, 2, 4, 4, 1, S::GL, 1, ring_depth(S::NL, 9 * S::CPT / S::GL), S::IL_L>(n, planes, legal, B, policy, value, s);
    return launch_cfg<MK, 256, 2, 2, 4, 1, S::GS, 1, ring_depth(S::NS, 9 * S::CPT / S::GS), S::IL_S>(n, planes, legal, B, policy, value, s);
  } else {
    static_assert(F == 64, "filters");
    if (tiling == 1)
      return launch_cfg<MK, 64, 1, 4, 2, 2, S::GL, 1, ring_depth(S::NL, 9 * S::CPT / S::GL), S::IL_L>(n, planes, legal, B, policy, value, s);
    if (tiling == 3)
      return launch_cfg<MK, 64, 1, 2, 2, 2, S::GM, 2, ring_depth(S::NM, 9 * S::CPT / S::GM), S::IL_M>(n, planes, legal, B, policy, value, s);
    return launch_cfg<MK, 64, 1, 2, 2, 1, S::GS, 2, ring_depth(S::NS, 9 * S::CPT / S::GS), S::IL_S>(n, planes, legal, B, policy, value, s);
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
  if (tiling == 3) return filters == 256 ? 1 : 2;
  return filters == 256 ? 2 : 4;
}

bool az_mfma_tiling_valid(int filters, int tiling) {
  return tiling == 1 || tiling == 2 || (tiling == 3 && filters != 256);
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
