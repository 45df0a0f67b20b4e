// Device helpers shared by the fused network kernels (gfx950): operand types
// and MFMA wrappers per element format, compile-time loops, bf16 / int8 / fp8
// conversions, activations and wave-wide reductions.  Private to the library:
// everything has internal linkage.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

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
constexpr int gcd_c(int a, int b) { return b == 0 ? a : gcd_c(b, a % b); }


template <int I, int N, class F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for<I + 1, N>(f);
  }
}

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
__device__ __forceinline__ float bf16_round(float f) { return __uint_as_float(bf16_bits(f) << 16); }

__device__ __forceinline__ float act_fn(float y, float cap) { return fminf(fmaxf(y, 0.0f), cap); }
__device__ __forceinline__ float med3(float x, float lo, float hi) {
  return __builtin_amdgcn_fmed3f(x, lo, hi);
}

// Code word of four values already on the code grid and in range (the
// hardware conversions then only re-encode them).
template <int MK>
__device__ __forceinline__ uint32_t pack_codes(float z0, float z1, float z2, float z3) {
  if constexpr (MK == MK_I8) {
    uint32_t w = __builtin_amdgcn_cvt_pk_u8_f32(z0, 0, 0u);
    w = __builtin_amdgcn_cvt_pk_u8_f32(z1, 1, w);
    w = __builtin_amdgcn_cvt_pk_u8_f32(z2, 2, w);
    return __builtin_amdgcn_cvt_pk_u8_f32(z3, 3, w);
  } else {
    int w = __builtin_amdgcn_cvt_pk_fp8_f32(z0, z1, 0, false);
    w = __builtin_amdgcn_cvt_pk_fp8_f32(z2, z3, w, true);
    return (uint32_t)w;
  }
}
// Requantisation in float64.  The next tensor's code is sat(rne(act(y) / a_out));
// the epilogues compute z = y / a_out from the exact accumulator with float64
// constants and round it here to the code grid (int8: the nearest integer; fp8:
// the nearest e4m3fn value; ties to even in both), then clamp the code to
// [0, hi], hi the tensor's largest code (rne(min(qmax, cap / a_out)) on the
// grid).  Rounding to the grid is monotone, so clamping the rounded value is
// rounding the clamped one.  float64 carries 53 bits, so a code can differ from
// exact arithmetic only within about 2^-45 of a tie.
//
// int8: adding 1.5 * 2^52 to z (|z| < 2^31) rounds it to an integer, to
// nearest even in the default rounding mode, and leaves that integer in the low
// 32 bits of the sum.
__device__ __forceinline__ int rne_i32(double z) {
  return (int)(uint32_t)__builtin_bit_cast(uint64_t, z + 6755399441055744.0);
}
// fp8: the spacing of e4m3 values around z is 2^(e-3), e = floor(log2 |z|) but at
// least -6 (subnormals share the spacing 2^-9)
__device__ __forceinline__ float e4m3_round_d(double z) {
  const int e = max(__builtin_amdgcn_frexp_exp(z) - 1, -6);
  return (float)__builtin_amdgcn_ldexp(__builtin_rint(__builtin_amdgcn_ldexp(z, 3 - e)), e - 3);
}
// min(max(x, lo), hi) for lo <= hi in one instruction (the compiler forms it
// only when it can prove lo <= hi)
__device__ __forceinline__ int med3_i32(int x, int lo, int hi) {
  int r;
  asm("v_med3_i32 %0, %1, %2, %3" : "=v"(r) : "v"(x), "v"(lo), "v"(hi));
  return r;
}
__device__ __forceinline__ double clamp_d(double z, double hi) { return __builtin_fmin(__builtin_fmax(z, 0.0), hi); }
// Code word of four requantised values.
template <int MK>
__device__ __forceinline__ uint32_t pack_codes_d(double z0, double z1, double z2, double z3, float hi) {
  if constexpr (MK == MK_I8) {
    const int h = (int)hi;  // >= 0
    const uint32_t c0 = med3_i32(rne_i32(z0), 0, h), c1 = med3_i32(rne_i32(z1), 0, h);
    const uint32_t c2 = med3_i32(rne_i32(z2), 0, h), c3 = med3_i32(rne_i32(z3), 0, h);
    return c0 | (c1 << 8) | (c2 << 16) | (c3 << 24);
  } else {
    return pack_codes<MK>(med3(e4m3_round_d(z0), 0.0f, hi), med3(e4m3_round_d(z1), 0.0f, hi),
                          med3(e4m3_round_d(z2), 0.0f, hi), med3(e4m3_round_d(z3), 0.0f, hi));
  }
}

// Value of byte R of a code word (codes of post-activation tensors are >= 0
// for int8; fp8 codes are decoded by the hardware conversion).
template <int MK, int R>
__device__ __forceinline__ float code_value(uint32_t x) {
  if constexpr (MK == MK_I8) return (float)((x >> (8 * R)) & 0xffu);  // codes are 0..127
  else return __builtin_amdgcn_cvt_f32_fp8((int)x, R);
}
template <int MK, int R>
__device__ __forceinline__ double code_value_d(uint32_t x) {
  if constexpr (MK == MK_I8) return (double)((x >> (8 * R)) & 0xffu);
  else return (double)__builtin_amdgcn_cvt_f32_fp8((int)x, R);
}

__device__ __forceinline__ float wave_max(float v) {
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

}  // namespace
