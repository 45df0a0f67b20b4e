// Host side of the C ABI: spec validation, weight rounding / quantisation,
// packing into the kernels' fragment order, device upload and dispatch.
//
// Packed weight streams (MFMA dtypes).  A 3x3 conv with C' input channels
// (the stem pads 20 -> 32) is the GEMM D[ch][sq] = sum_k W[ch][k] X[k][sq] with
// k = tap * C' + c, tap = 3*dy + dx.  With KS the reduction length of one MFMA
// (bf16 16, int8 32, fp8 64) the stream holds, for every K step s and every
// 32-channel block mb, one 64-lane fragment; lane l carries
//   W[mb*32 + l%32][s*KS + (KS/2)*(l/32) + t],  t = 0 .. KS/2-1,
// contiguously (16 bytes for bf16 and int8, 32 for fp8), so that a wave loads
// a fragment with one fully coalesced read.  The B-operand (activation) lanes
// use the same k slots, so the pairing of A and B k values matches by
// construction.  Order: stem (bf16), then the 2*blocks residual convs, then
// the head: 96 rows (policy planes, value 1x1 conv row, zero rows), K = F.
//
// The deployed network (from-to policy, WDL value, global pooling) pads the
// stem to 64 input channels, packs the second convolution of a pooling block
// ([F][Fr][3][3]) with zero weights for input channels Fr..F-1, and packs its
// heads as described in az_dep_kernel.h.
#include "../../include/az.h"
#include "az_internal.h"

#include <math.h>
#include <stdarg.h>
#include <stddef.h>
#include <stdlib.h>
#include <stdio.h>
#include <string.h>

#include <atomic>
#include <new>
#include <string>
#include <vector>

struct az_net {
  az_layer_spec spec;
  int dtype;
  int device;
  int tiling;  // 0 = chosen per batch
  int cus;     // compute units of the device
  void* dmem;
  size_t dbytes;
  AzDevNet dn;
};

namespace {

thread_local std::string g_err;

int fail(int status, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return status;
}

int hip_fail(hipError_t e, const char* what) {
  const int st = (e == hipErrorOutOfMemory || e == hipErrorMemoryAllocation) ? AZ_ERR_NOMEM
                                                                            : AZ_ERR_DEVICE;
  return fail(st, "%s: %s", what, hipGetErrorString(e));
}

// Bytes of a version-1 spec: the fields before pool_every.
constexpr size_t kSpecV1Bytes = offsetof(az_layer_spec, pool_every);

// Copies a caller's spec into the current layout (version-1 callers pass the
// first nine fields only: the move-plane network with the tanh value head).
bool normalize_spec(const az_layer_spec* in, az_layer_spec* out) {
  if (!in) return false;
  if (in->abi_version == 1) {
    memset(out, 0, sizeof *out);
    memcpy(out, in, kSpecV1Bytes);
    out->value_channels = 1;
  } else if (in->abi_version == 2) {
    *out = *in;
  } else {
    return false;
  }
  out->abi_version = AZ_ABI_VERSION;
  return true;
}

bool is_pool_block(const az_layer_spec& s, int j) {
  return s.pool_every > 0 && j % s.pool_every == s.pool_every - 1;
}

bool is_deployed(const az_layer_spec& s) {
  return s.policy_head == AZ_POLICY_FROMTO || s.value_head == AZ_VALUE_WDL || s.pool_every > 0;
}

bool spec_well_formed(const az_layer_spec& s) {
  if (!(s.in_planes >= 1 && s.blocks >= 1 && s.filters >= 1 && s.value_hidden >= 1 &&
        (s.value_conv_relu == 0 || s.value_conv_relu == 1) && s.act_cap >= 0.0f && isfinite(s.act_cap) &&
        s.max_batch >= 1 && s.pool_every >= 0))
    return false;
  if (s.policy_head == AZ_POLICY_PLANES) {
    if (s.policy_planes < 1 || s.token_dim != 0) return false;
  } else if (s.policy_head == AZ_POLICY_FROMTO) {
    if (s.policy_planes != 0 || s.token_dim < 1) return false;
  } else {
    return false;
  }
  if (s.value_head == AZ_VALUE_TANH) {
    if (s.value_channels != 1) return false;
  } else if (s.value_head == AZ_VALUE_WDL) {
    if (s.value_channels < 1) return false;
  } else {
    return false;
  }
  return s.pool_every == 0 || s.filters % 4 == 0;
}

int check_spec(const az_layer_spec& s, int dtype) {
  if (!spec_well_formed(s)) return fail(AZ_ERR_INVALID_ARG, "malformed az_layer_spec");
  if (dtype < AZ_F32 || dtype > AZ_FP8_E4M3) return fail(AZ_ERR_INVALID_ARG, "unknown dtype %d", dtype);
  if (s.blocks > 64) return fail(AZ_ERR_UNSUPPORTED, "blocks %d > 64", s.blocks);
  if (s.value_hidden > 512) return fail(AZ_ERR_UNSUPPORTED, "value_hidden %d > 512", s.value_hidden);
  if (s.max_batch > (1 << 20)) return fail(AZ_ERR_UNSUPPORTED, "max_batch %d > 2^20", s.max_batch);
  if (is_deployed(s)) {
    if (s.policy_head != AZ_POLICY_FROMTO || s.value_head != AZ_VALUE_WDL)
      return fail(AZ_ERR_UNSUPPORTED, "global pooling, the from-to policy and the WDL value head come together");
    if (dtype != AZ_BF16 && dtype != AZ_INT8) return fail(AZ_ERR_UNSUPPORTED, "the deployed network runs in AZ_BF16 or AZ_INT8");
    if (s.filters != 160) return fail(AZ_ERR_UNSUPPORTED, "the deployed network needs filters 160, got %d", s.filters);
    if (s.token_dim != AZ_DEP_TOKEN) return fail(AZ_ERR_UNSUPPORTED, "token_dim %d != %d", s.token_dim, AZ_DEP_TOKEN);
    if (s.value_channels > AZ_DEP_EMB_ROWS - AZ_DEP_TOKEN)
      return fail(AZ_ERR_UNSUPPORTED, "value_channels %d > %d", s.value_channels, AZ_DEP_EMB_ROWS - AZ_DEP_TOKEN);
    if (s.in_planes > AZ_DEP_MAX_IN_PLANES) return fail(AZ_ERR_UNSUPPORTED, "in_planes %d > %d", s.in_planes, AZ_DEP_MAX_IN_PLANES);
    return AZ_OK;
  }
  if (s.in_planes > AZ_MAX_IN_PLANES) return fail(AZ_ERR_UNSUPPORTED, "in_planes %d > %d", s.in_planes, AZ_MAX_IN_PLANES);
  if (s.policy_planes > AZ_MAX_POLICY) return fail(AZ_ERR_UNSUPPORTED, "policy_planes %d > %d", s.policy_planes, AZ_MAX_POLICY);
  if (dtype == AZ_F32) {
    if (s.filters % 8 != 0 || s.filters > 256) return fail(AZ_ERR_UNSUPPORTED, "AZ_F32 needs filters a multiple of 8 up to 256, got %d", s.filters);
  } else if (!az_mfma_supported(dtype, s.filters)) {
    return fail(AZ_ERR_UNSUPPORTED, "dtype %d needs filters in {64, 128, 256}, got %d", dtype, s.filters);
  }
  return AZ_OK;
}

size_t weight_count(const az_layer_spec& s) {
  const size_t C = s.in_planes, F = s.filters, P = s.policy_planes, H = s.value_hidden;
  const size_t g = s.pool_every > 0 ? F / 4 : 0, Fr = F - g, D = s.token_dim, V = s.value_channels;
  size_t n = F * C * 9 + F;
  for (int j = 0; j < s.blocks; ++j)
    n += F * F * 9 + F + (is_pool_block(s, j) ? Fr * 2 * g + F * Fr * 9 + F : F * F * 9 + F);
  n += s.policy_head == AZ_POLICY_FROMTO ? D * F + D + 2 * (D * D + D) + 4 * D : P * F + P;
  n += s.value_head == AZ_VALUE_WDL ? V * F + V + H * V * 64 + H + 3 * H + 3 : F + 1 + H * 64 + H + H + 1;
  return n;
}

// Offsets of the arrays inside the canonical blob.
struct BlobView {
  const float *stem_w, *stem_b, *pol_w, *pol_b, *val_w, *val_b, *fc1_w, *fc1_b, *fc2_w, *fc2_b;
  std::vector<const float*> w, b;  // residual conv n = 2j (first) and 2j+1 (second)
  std::vector<const float*> pool;  // per block: Wg [Fr][2g] or NULL
  // from-to head
  const float *emb_w = nullptr, *emb_b = nullptr, *q_w = nullptr, *q_b = nullptr, *k_w = nullptr,
              *k_b = nullptr, *p_w = nullptr;
};

BlobView view(const az_layer_spec& s, const float* blob) {
  const size_t C = s.in_planes, F = s.filters, P = s.policy_planes, H = s.value_hidden;
  const size_t g = s.pool_every > 0 ? F / 4 : 0, Fr = F - g, D = s.token_dim, V = s.value_channels;
  BlobView v;
  const float* q = blob;
  v.stem_w = q; q += F * C * 9;
  v.stem_b = q; q += F;
  for (int j = 0; j < s.blocks; ++j) {
    const bool pool = is_pool_block(s, j);
    v.w.push_back(q); q += F * F * 9;
    v.b.push_back(q); q += F;
    v.pool.push_back(pool ? q : nullptr);
    if (pool) q += Fr * 2 * g;
    v.w.push_back(q); q += F * (pool ? Fr : F) * 9;
    v.b.push_back(q); q += F;
  }
  if (s.policy_head == AZ_POLICY_FROMTO) {
    v.emb_w = q; q += D * F;
    v.emb_b = q; q += D;
    v.q_w = q; q += D * D;
    v.q_b = q; q += D;
    v.k_w = q; q += D * D;
    v.k_b = q; q += D;
    v.p_w = q; q += 4 * D;
    v.pol_w = v.pol_b = nullptr;
  } else {
    v.pol_w = q; q += P * F;
    v.pol_b = q; q += P;
  }
  const size_t VR = s.value_head == AZ_VALUE_WDL ? V : 1;
  v.val_w = q; q += VR * F;
  v.val_b = q; q += VR;
  v.fc1_w = q; q += H * VR * 64;
  v.fc1_b = q; q += H;
  v.fc2_w = q; q += (s.value_head == AZ_VALUE_WDL ? 3 : 1) * H;
  v.fc2_b = q; q += s.value_head == AZ_VALUE_WDL ? 3 : 1;
  return v;
}

uint16_t bf16_rne(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  if ((u & 0x7f800000u) == 0x7f800000u) return (uint16_t)((u >> 16) | ((u & 0xffffu) ? 0x40u : 0u));
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

int8_t quant_i8(double v) {
  double r = nearbyint(v);  // default rounding mode: to nearest, ties to even
  if (r > 127.0) r = 127.0;
  if (r < -127.0) r = -127.0;
  return (int8_t)r;
}

// OCP fp8 e4m3fn code of v: nearest value, ties to even, saturating to +-448.
uint8_t quant_e4m3(double v) {
  const uint8_t sign = signbit(v) ? 0x80 : 0x00;
  const double a = fabs(v);
  if (!(a > 0.0)) return sign;
  if (a >= 448.0) return sign | 0x7e;
  int ex;
  frexp(a, &ex);  // a = m * 2^ex, m in [0.5, 1)
  int e = ex - 1;
  if (e < -6) e = -6;
  const double step = ldexp(1.0, e - 3);
  double r = nearbyint(a / step) * step;
  if (r > 448.0) r = 448.0;
  if (r == 0.0) return sign;
  frexp(r, &ex);
  e = ex - 1;
  if (e < -6) return sign | (uint8_t)(r / ldexp(1.0, -9));  // subnormal: m * 2^-9
  const int mant = (int)((r / ldexp(1.0, e) - 1.0) * 8.0);
  return sign | (uint8_t)(((e + 7) << 3) | mant);
}

// Value of an e4m3fn code (finite codes only).
float e4m3_value(uint8_t c) {
  const int e = (c >> 3) & 15, m = c & 7;
  const double v = e == 0 ? ldexp((double)m, -9) : ldexp(1.0 + m / 8.0, e - 7);
  return (float)((c & 0x80) ? -v : v);
}

enum Kind { K_BF16 = 0, K_I8 = 1, K_F8 = 2 };

// Packs a 3x3 conv W[F][Cin][3][3] (padded to Cp input channels) into A fragments.
void pack_conv(const float* W, const float* wscale, int F, int Cin, int Cp, Kind kind,
               std::vector<uint8_t>& out) {
  const int KS = kind == K_BF16 ? 16 : kind == K_I8 ? 32 : 64;
  const int es = kind == K_BF16 ? 2 : 1;
  const int half = KS / 2, FB = half * es, nMB = F / 32, S = 9 * Cp / KS;
  const size_t base = out.size();
  out.resize(base + (size_t)S * nMB * 64 * FB);
  uint8_t* o = out.data() + base;
  for (int s = 0; s < S; ++s)
    for (int mb = 0; mb < nMB; ++mb)
      for (int l = 0; l < 64; ++l) {
        const int ch = mb * 32 + l % 32;
        uint8_t* dst = o + ((size_t)(s * nMB + mb) * 64 + l) * FB;
        for (int t = 0; t < half; ++t) {
          const int k = s * KS + half * (l / 32) + t, tap = k / Cp, c = k % Cp;
          const float v = c < Cin ? W[((size_t)ch * Cin + c) * 9 + tap] : 0.0f;
          if (kind == K_BF16) {
            const uint16_t h = bf16_rne(v);
            memcpy(dst + 2 * t, &h, 2);
          } else {
            // float64 quotient of two float32 values: it rounds only off the
            // code grid's ties, so the code is that of the exact quotient
            const double x = (double)v / (double)wscale[ch];
            dst[t] = kind == K_I8 ? (uint8_t)quant_i8(x) : quant_e4m3(x);
          }
        }
      }
}

void pack_head(const BlobView& v, int F, int P, std::vector<uint8_t>& out) {
  const int S = F / 16;
  const size_t base = out.size();
  out.resize(base + (size_t)S * 3 * 64 * 16);
  uint8_t* o = out.data() + base;
  for (int s = 0; s < S; ++s)
    for (int mb = 0; mb < 3; ++mb)
      for (int l = 0; l < 64; ++l) {
        const int row = mb * 32 + l % 32;
        for (int t = 0; t < 8; ++t) {
          const int k = s * 16 + 8 * (l / 32) + t;
          const float w = row < P ? v.pol_w[(size_t)row * F + k] : row == P ? v.val_w[k] : 0.0f;
          const uint16_t h = bf16_rne(w);
          memcpy(o + ((size_t)(s * 3 + mb) * 64 + l) * 16 + 2 * t, &h, 2);
        }
      }
}

// ---- deployed network -------------------------------------------------------
//
// bf16 A fragments of a row-major matrix M[rows][K] (rows padded with zeros to
// nMB*32, K a multiple of 16): fragment (s, mb), lane l holds
// M[mb*32 + l%32][kperm(s, l/32, t)], t = 0..7.  The plain order is
// kperm = s*16 + 8*(l/32) + t.
template <class KPerm>
void pack_rows_bf16(const float* M, int rows, int K, int nMB, KPerm kperm, std::vector<uint8_t>& out) {
  const int S = K / 16;
  const size_t base = out.size();
  out.resize(base + (size_t)S * nMB * 64 * 16);
  uint8_t* o = out.data() + base;
  for (int s = 0; s < S; ++s)
    for (int mb = 0; mb < nMB; ++mb)
      for (int l = 0; l < 64; ++l) {
        const int row = mb * 32 + l % 32;
        for (int t = 0; t < 8; ++t) {
          const float w = row < rows ? M[(size_t)row * K + kperm(s, l / 32, t)] : 0.0f;
          const uint16_t h = bf16_rne(w);
          memcpy(o + ((size_t)(s * nMB + mb) * 64 + l) * 16 + 2 * t, &h, 2);
        }
      }
}

// Row index held at position p (0..63) of the accumulators of lane half lhi of
// an output with 128 rows (four 32-row blocks): block p/16, register v = p%16,
// row 32*(p/16) + 8*(v/4) + 4*lhi + v%4.  The token, query and key
// accumulators feed the next products directly as operands: K step s, lane
// half lhi, slot t carries position 8*s + t, so the weights that multiply them
// are packed with their K dimension in this order.
int acc_row(int s, int lhi, int t) {
  const int p = 8 * s + t, v = p % 16;
  return 32 * (p / 16) + 8 * (v / 4) + 4 * lhi + v % 4;
}

// Action table of the from-to policy: origin-destination pairs on a common
// row, column or diagonal or a knight's jump apart, ascending (origin,
// destination); then the promotions from row 6 to row 7 at most one column
// over, pieces queen, rook, bishop, knight, ascending (origin, destination,
// piece).  Entry: origin*64 + destination, plus (column*4 + piece + 1) << 12
// for a promotion (its offset O[column][piece]).
std::vector<uint32_t> fromto_actions() {
  std::vector<uint32_t> a;
  for (int f = 0; f < 64; ++f)
    for (int t = 0; t < 64; ++t) {
      if (t == f) continue;
      const int dr = abs(t / 8 - f / 8), dc = abs(t % 8 - f % 8);
      if (dr == 0 || dc == 0 || dr == dc || (dr == 1 && dc == 2) || (dr == 2 && dc == 1))
        a.push_back((uint32_t)(f * 64 + t));
    }
  for (int fc = 0; fc < 8; ++fc)
    for (int tc = fc > 0 ? fc - 1 : 0; tc <= (fc < 7 ? fc + 1 : 7); ++tc)
      for (int k = 0; k < 4; ++k)
        a.push_back((uint32_t)((48 + fc) * 64 + 56 + tc) | ((uint32_t)(tc * 4 + k + 1) << 12));
  return a;
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

// Measured on MI355X (20x128 and 24x256 networks): one board per workgroup wins
// below a few hundred boards; at 1024 boards the four-board large tiling wins
// for bf16 and fp8, and the two-board medium tiling (two workgroups per compute
// unit) ties with it for int8.
//
// Deployed network: the tiling with the shorter estimated time, rounds x time
// per round.  A round is one board per compute unit with four waves per board,
// and four (int8) or three (bf16, LDS-bound) boards per compute unit with one
// wave per board; a round of the latter takes 2.5x (int8: ~370 against ~150 us)
// or 2.8x (bf16: ~630 against ~225 us) as long as one of the former (14x160 on
// MI355X).
int choose_dep_tiling(const az_net* n, int B) {
  const bool i8 = n->dtype == AZ_INT8;
  const long per1 = (long)n->cus * (i8 ? 4 : 3), per2 = n->cus;
  const long r1 = (B + per1 - 1) / per1, r2 = (B + per2 - 1) / per2;
  return r2 * 10 < r1 * (i8 ? 25 : 28) ? 2 : 1;
}

int choose_tiling(const az_net* n, int B) {
  if (n->dtype == AZ_F32) return 0;
  if (n->tiling) return n->tiling;
  if (is_deployed(n->spec)) return choose_dep_tiling(n, B);
  const int F = n->spec.filters;
  if (B < 512) return 2;
  // Measured on 20x128 (us per batch, large / one-board / medium tiling):
  // int8 768 boards 293 / 283 / 295, 896 boards 303 / 342 / 311, 1,024 boards
  // 327 / 368 / 338; bf16 640 boards 487 / 459 / 458, 768 boards 495 / 510 / 512.
  // fp8: 640 boards 335 / 293 / 314, 768 boards 337 / 310 / 326, 896 boards
  // 340 / 384 / 337, 1,024 boards 350 / 402 / 357.
  if (n->dtype == AZ_INT8) return B <= 768 ? 2 : 1;
  if (n->dtype == AZ_BF16) return B >= 768 ? 1 : 2;
  if (B <= 768) return 2;
  if (B >= 1024) return 1;
  return az_mfma_tiling_valid(F, 3) ? 3 : 1;
}

}  // namespace

// Counted allocations (see az_internal.h).  g_fail_in > 0 counts down to the
// allocation that is made to fail.
namespace {
std::atomic<int64_t> g_live{0};
std::atomic<int32_t> g_fail_in{0};

bool injected_failure() {
  int32_t c = g_fail_in.load();
  while (c > 0 && !g_fail_in.compare_exchange_weak(c, c - 1)) {
  }
  return c == 1;
}
}  // namespace

hipError_t az_dev_malloc(void** ptr, size_t bytes) {
  *ptr = nullptr;
  if (injected_failure()) return hipErrorOutOfMemory;
  const hipError_t e = hipMalloc(ptr, bytes);
  if (e == hipSuccess) ++g_live;
  return e;
}
void az_dev_free(void* ptr) {
  if (!ptr) return;
  (void)hipFree(ptr);
  --g_live;
}
hipError_t az_host_malloc(void** ptr, size_t bytes) {
  *ptr = nullptr;
  if (injected_failure()) return hipErrorOutOfMemory;
  const hipError_t e = hipHostMalloc(ptr, bytes, hipHostMallocDefault);
  if (e == hipSuccess) ++g_live;
  return e;
}
void az_host_free(void* ptr) {
  if (!ptr) return;
  (void)hipHostFree(ptr);
  --g_live;
}

// Records the detail of a failure for az_last_error() (used by the other
// translation units of the library).
int az_fail(int status, const char* detail) { return fail(status, "%s", detail); }

const az_layer_spec& az_net_spec(const az_net* n) { return n->spec; }
int az_spec_moves(const az_layer_spec& s) {
  return s.policy_head == AZ_POLICY_FROMTO ? AZ_FROMTO_ACTIONS : s.policy_planes * AZ_SQUARES;
}
int az_net_device(const az_net* n) { return n->device; }

extern "C" {

size_t az_weight_count(const az_layer_spec* spec) {
  az_layer_spec s;
  if (!normalize_spec(spec, &s) || !spec_well_formed(s)) return 0;
  return weight_count(s);
}

const char* az_status_string(int status) {
  switch (status) {
    case AZ_OK: return "ok";
    case AZ_ERR_INVALID_ARG: return "invalid argument";
    case AZ_ERR_UNSUPPORTED: return "unsupported network or dtype";
    case AZ_ERR_NOMEM: return "device out of memory";
    case AZ_ERR_DEVICE: return "HIP device error";
    default: return "unknown status";
  }
}

const char* az_last_error(void) { return g_err.c_str(); }

void az_debug_fail_allocation(int32_t n) { g_fail_in.store(n > 0 ? n : 0); }

int64_t az_debug_live_allocations(void) { return g_live.load(); }

int az_net_load(const az_layer_spec* spec_in, const float* weights, size_t n_weights, int32_t dtype,
                const float* w_scales, size_t n_w_scales, const float* act_scales,
                size_t n_act_scales, az_net** out) {
  g_err.clear();
  if (!out || !weights) return fail(AZ_ERR_INVALID_ARG, "NULL weights or out pointer");
  az_layer_spec s;
  if (!normalize_spec(spec_in, &s)) return fail(AZ_ERR_INVALID_ARG, "malformed az_layer_spec");
  int st = check_spec(s, dtype);
  if (st != AZ_OK) return st;
  if (n_weights != weight_count(s))
    return fail(AZ_ERR_INVALID_ARG, "n_weights %zu, the spec needs %zu", n_weights, weight_count(s));
  const int F = s.filters, NB = s.blocks, P = s.policy_planes, H = s.value_hidden, Cin = s.in_planes;
  const bool quant = dtype == AZ_INT8 || dtype == AZ_FP8_E4M3;
  const bool dep = is_deployed(s);
  if (quant) {
    if (!w_scales || n_w_scales != (size_t)2 * NB * F)
      return fail(AZ_ERR_INVALID_ARG, "need %d weight scales, got %zu", 2 * NB * F, n_w_scales);
    if (!act_scales || n_act_scales != (size_t)2 * NB + 1)
      return fail(AZ_ERR_INVALID_ARG, "need %d activation scales, got %zu", 2 * NB + 1, n_act_scales);
    for (size_t i = 0; i < n_w_scales; ++i)
      if (!(w_scales[i] > 0.0f) || !isfinite(w_scales[i])) return fail(AZ_ERR_INVALID_ARG, "weight scale %zu not positive finite", i);
    for (size_t i = 0; i < n_act_scales; ++i)
      if (!(act_scales[i] > 0.0f) || !isfinite(act_scales[i])) return fail(AZ_ERR_INVALID_ARG, "activation scale %zu not positive finite", i);
  } else if (w_scales || n_w_scales || act_scales || n_act_scales) {
    return fail(AZ_ERR_INVALID_ARG, "scales are only taken for AZ_INT8 and AZ_FP8_E4M3");
  }

  const BlobView v = view(s, weights);
  const int g = s.pool_every > 0 ? F / 4 : 0, Fr = F - g, V = s.value_channels, D = s.token_dim;
  std::vector<uint8_t> stem, tower, head, emb, qw, kw, pw;
  std::vector<float> bias, qhi, head_b, fc2w, head_sc, head_bc, fc1t;
  std::vector<double> qmul, qbias, qres, qext, pool_m, pool_b, pool_cinv;
  std::vector<float> emb_sc, emb_bc, wfc1t;
  std::vector<float> pool_wt;
  std::vector<uint32_t> actions;
  const float hs = quant ? act_scales[2 * NB] : 1.0f;
  try {
    bias.resize((size_t)(1 + 2 * NB) * F);
    memcpy(bias.data(), v.stem_b, F * sizeof(float));
    for (int n = 0; n < 2 * NB; ++n) memcpy(bias.data() + (size_t)(1 + n) * F, v.b[n], F * sizeof(float));
    if (!dep) {
      head_b.assign(AZ_HEAD_ROWS, 0.0f);
      fc2w.assign(v.fc2_w, v.fc2_w + H);
      for (int i = 0; i < P; ++i) head_b[i] = v.pol_b[i];
      head_b[P] = v.val_b[0];
      // MFMA kernels: every head row r stores fma(acc, head_sc[r], head_bc[r]); policy
      // rows come out pre-scaled by log2(e) for the exp2 softmax, the value row P
      // unscaled, padding rows zero.  Products rounded once to float32.
      const float log2e = 1.4426950408889634f;
      head_sc.assign(AZ_HEAD_ROWS, 0.0f);
      head_bc.assign(AZ_HEAD_ROWS, 0.0f);
      for (int i = 0; i < P; ++i) {
        head_sc[i] = hs * log2e;
        head_bc[i] = v.pol_b[i] * log2e;
      }
      head_sc[P] = hs;
      head_bc[P] = v.val_b[0];
      // fc1 for the MFMA kernels as [64/4][H][4]: lane k of a wave reads
      // W1[k][4s .. 4s+3] at ((s * H + k) * 4), so a wave's float4 loads are contiguous.
      fc1t.resize((size_t)H * 64);
      for (int k = 0; k < H; ++k)
        for (int c = 0; c < 64; ++c) fc1t[((size_t)(c / 4) * H + k) * 4 + (c % 4)] = v.fc1_w[(size_t)k * 64 + c];
    }
    if (dtype == AZ_F32) {
      // fp32 kernel: convs as [F/8][C][9][8] and heads as [ceil((P+1)/8)][F][8], so
      // that the eight output channels (rows) a thread accumulates at one (input
      // channel, tap) are one contiguous 32-byte load
      auto pack8 = [](const float* W, int Fo, int C, std::vector<uint8_t>& out) {
        const size_t base = out.size();
        out.resize(base + (size_t)Fo * C * 9 * 4);
        float* o = reinterpret_cast<float*>(out.data() + base);
        for (int fb = 0; fb < Fo / 8; ++fb)
          for (int c = 0; c < C; ++c)
            for (int t = 0; t < 9; ++t)
              for (int j = 0; j < 8; ++j)
                o[(((size_t)fb * C + c) * 9 + t) * 8 + j] = W[((size_t)(fb * 8 + j) * C + c) * 9 + t];
      };
      pack8(v.stem_w, F, Cin, stem);
      for (int n = 0; n < 2 * NB; ++n) pack8(v.w[n], F, F, tower);
      const int RB8 = (P + 1 + 7) / 8;
      head.assign((size_t)RB8 * F * 8 * 4, 0);
      float* h = reinterpret_cast<float*>(head.data());
      for (int rb = 0; rb < RB8; ++rb)
        for (int f = 0; f < F; ++f)
          for (int j = 0; j < 8; ++j) {
            const int row = rb * 8 + j;
            h[((size_t)rb * F + f) * 8 + j] = row < P ? v.pol_w[(size_t)row * F + f] : row == P ? v.val_w[f] : 0.0f;
          }
    } else {
      pack_conv(v.stem_w, nullptr, F, Cin, dep ? AZ_DEP_MAX_IN_PLANES : 32, K_BF16, stem);
      const Kind kind = dtype == AZ_BF16 ? K_BF16 : dtype == AZ_INT8 ? K_I8 : K_F8;
      for (int n = 0; n < 2 * NB; ++n) {
        // the second convolution of a pooling block reads the Fr regular channels
        const int cin = (n % 2 == 1 && is_pool_block(s, n / 2)) ? Fr : F;
        pack_conv(v.w[n], quant ? w_scales + (size_t)n * F : nullptr, F, cin, F, kind, tower);
      }
      if (!dep) pack_head(v, F, P, head);
      if (quant) {
        // Requantisation constants in float64: an output's code is
        // rne(clamp(acc * qmul + qbias (+ qres * residual code), 0, qhi)).
        const int K = 2 * NB + 1;
        const double qmax = dtype == AZ_INT8 ? 127.0 : 448.0;
        std::vector<double> a(act_scales, act_scales + K);
        qmul.resize((size_t)K * F);
        qbias.resize((size_t)K * F);
        qres.assign(K, 0.0);
        qhi.resize(K);
        for (int f = 0; f < F; ++f) {
          qmul[f] = 1.0 / a[0];
          qbias[f] = (double)v.stem_b[f] / a[0];
        }
        for (int n = 0; n < 2 * NB; ++n)
          for (int f = 0; f < F; ++f) {
            qmul[(size_t)(1 + n) * F + f] = a[n] * (double)w_scales[(size_t)n * F + f] / a[n + 1];
            qbias[(size_t)(1 + n) * F + f] = (double)v.b[n][f] / a[n + 1];
          }
        for (int k = 0; k < K; ++k) {
          if (k >= 2 && k % 2 == 0) qres[k] = a[k - 2] / a[k];
          // the largest code: min(qmax, cap / a[k]) rounded to the grid
          double c = s.act_cap > 0.0f ? (double)s.act_cap / a[k] : qmax;
          if (c > qmax) c = qmax;
          qhi[k] = dtype == AZ_INT8 ? (float)quant_i8(c) : e4m3_value(quant_e4m3(c));
        }
        qext.resize((size_t)2 * K);
        for (int k = 0; k < K; ++k) {
          qext[2 * k] = qres[k];
          qext[2 * k + 1] = qhi[k];
        }
      }
      if (dep) {
        // global pooling (int8): the pooled channels' activation
        // act(acc * pool_m + pool_b) and the factor of the projected context c in
        // the regular channels' requantisation; bf16 pools act(acc + b1) itself
        if (quant) {
          pool_m.assign((size_t)2 * NB * F, 0.0);
          pool_b.assign((size_t)2 * NB * F, 0.0);
          pool_cinv.assign((size_t)2 * NB, 0.0);
        }
        for (int j = 0; j < NB; ++j) {
          if (!is_pool_block(s, j)) continue;
          const int n = 2 * j;
          if (quant) {
            for (int f = 0; f < F; ++f) {
              pool_b[(size_t)n * F + f] = v.b[n][f];
              pool_m[(size_t)n * F + f] = (double)act_scales[n] * (double)w_scales[(size_t)n * F + f];
            }
            pool_cinv[n] = 1.0 / (double)act_scales[n + 1];
          }
          // Wg as [2g/4][AZ_DEP_POOL_OPAD][4] (outputs padded with zeros): lane o of
          // a wave loads Wg[o][4s .. 4s+3] at ((s * OPAD + o) * 4), so the wave's
          // float4 loads are contiguous
          const size_t base = pool_wt.size();
          pool_wt.resize(base + (size_t)2 * g * AZ_DEP_POOL_OPAD, 0.0f);
          for (int i = 0; i < 2 * g; ++i)
            for (int o = 0; o < Fr; ++o)
              pool_wt[base + ((size_t)(i / 4) * AZ_DEP_POOL_OPAD + o) * 4 + i % 4] = v.pool[j][(size_t)o * 2 * g + i];
        }
        // embedding: D token rows (We) then V value rows (Wv), K = F, plain K order
        std::vector<float> E((size_t)AZ_DEP_EMB_ROWS * F, 0.0f);
        memcpy(E.data(), v.emb_w, (size_t)D * F * sizeof(float));
        memcpy(E.data() + (size_t)D * F, v.val_w, (size_t)V * F * sizeof(float));
        pack_rows_bf16(E.data(), D + V, F, AZ_DEP_EMB_ROWS / 32,
                       [](int st, int lhi, int t) { return st * 16 + 8 * lhi + t; }, emb);
        emb_sc.assign(AZ_DEP_EMB_ROWS, 0.0f);
        emb_bc.assign(AZ_DEP_EMB_ROWS, 0.0f);
        for (int r = 0; r < D + V; ++r) {
          emb_sc[r] = hs;
          emb_bc[r] = r < D ? v.emb_b[r] : v.val_b[r - D];
        }
        // query, key and promotion weights: K dimension in the accumulators' order
        pack_rows_bf16(v.q_w, D, D, D / 32, acc_row, qw);
        pack_rows_bf16(v.k_w, D, D, D / 32, acc_row, kw);
        pack_rows_bf16(v.p_w, 4, D, 1, acc_row, pw);
        // WDL: fc1 transposed to [V*64][H] so that lane k's loads are contiguous
        wfc1t.resize((size_t)V * 64 * H);
        for (int k = 0; k < H; ++k)
          for (int i = 0; i < V * 64; ++i) wfc1t[(size_t)i * H + k] = v.fc1_w[(size_t)k * V * 64 + i];
        actions = fromto_actions();
        if (actions.size() != AZ_FROMTO_ACTIONS) return fail(AZ_ERR_DEVICE, "action table has %zu entries", actions.size());
        actions.resize(AZ_DEP_ACTION_SLOTS, 0u);
      }
    }
  } catch (const std::bad_alloc&) {
    return fail(AZ_ERR_NOMEM, "host allocation failed while packing weights");
  }

  // One device allocation, 256-byte aligned sections.
  struct Sec { const void* src; size_t bytes; size_t off; };
  const size_t VH = dep ? (size_t)V * 64 * H : (size_t)H * 64;
  std::vector<Sec> secs = {
      {stem.data(), stem.size(), 0}, {tower.data(), tower.size(), 0}, {head.data(), head.size(), 0},
      {bias.data(), bias.size() * 4, 0}, {qmul.data(), qmul.size() * 8, 0},
      {qres.data(), qres.size() * 8, 0}, {qhi.data(), qhi.size() * 4, 0},
      {head_b.data(), head_b.size() * 4, 0}, {dep ? nullptr : v.fc1_w, dep ? 0 : VH * 4, 0},
      {v.fc1_b, (size_t)H * 4, 0}, {dep ? (const void*)v.fc2_w : fc2w.data(), (dep ? 3 : 1) * (size_t)H * 4, 0},
      {head_sc.data(), head_sc.size() * 4, 0}, {head_bc.data(), head_bc.size() * 4, 0},
      {fc1t.data(), fc1t.size() * 4, 0},
      // deployed network
      {emb.data(), emb.size(), 0}, {qw.data(), qw.size(), 0}, {kw.data(), kw.size(), 0},
      {pw.data(), pw.size(), 0}, {emb_sc.data(), emb_sc.size() * 4, 0}, {emb_bc.data(), emb_bc.size() * 4, 0},
      {dep ? v.q_b : nullptr, dep ? (size_t)D * 4 : 0, 0}, {dep ? v.k_b : nullptr, dep ? (size_t)D * 4 : 0, 0},
      {pool_wt.data(), pool_wt.size() * 4, 0}, {pool_m.data(), pool_m.size() * 8, 0},
      {pool_b.data(), pool_b.size() * 8, 0}, {pool_cinv.data(), pool_cinv.size() * 8, 0},
      {actions.data(), actions.size() * 4, 0}, {wfc1t.data(), wfc1t.size() * 4, 0},
      {qbias.data(), qbias.size() * 8, 0}, {qext.data(), qext.size() * 8, 0}};
  size_t total = 0;
  for (auto& sc : secs) { sc.off = total; total += align256(sc.bytes); }

  int dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return hip_fail(e, "hipDeviceGetAttribute");
  void* dmem = nullptr;
  e = az_dev_malloc(&dmem, total);
  if (e != hipSuccess) { (void)hipGetLastError(); return hip_fail(e, "hipMalloc of the weights"); }
  for (auto& sc : secs) {
    if (!sc.bytes) continue;
    e = hipMemcpy(static_cast<uint8_t*>(dmem) + sc.off, sc.src, sc.bytes, hipMemcpyHostToDevice);
    if (e != hipSuccess) { az_dev_free(dmem); return hip_fail(e, "hipMemcpy of the weights"); }
  }
  az_net* net = new (std::nothrow) az_net;
  if (!net) { az_dev_free(dmem); return fail(AZ_ERR_NOMEM, "host allocation of the handle failed"); }
  auto at = [&](int i) { return secs[i].bytes ? static_cast<uint8_t*>(dmem) + secs[i].off : nullptr; };
  auto atf = [&](int i) { return reinterpret_cast<const float*>(at(i)); };
  auto atd = [&](int i) { return reinterpret_cast<const double*>(at(i)); };
  net->spec = s;
  net->dtype = dtype;
  net->device = dev;
  net->tiling = 0;
  net->cus = cus > 0 ? cus : 1;
  net->dmem = dmem;
  net->dbytes = total;
  AzDevNet& d = net->dn;
  memset(&d, 0, sizeof d);
  d.in_planes = Cin;
  d.blocks = NB;
  d.filters = F;
  d.policy_planes = P;
  d.value_hidden = H;
  d.value_conv_relu = s.value_conv_relu;
  d.act_cap = s.act_cap > 0.0f ? s.act_cap : INFINITY;
  d.head_scale = hs;
  d.stem_w = at(0);
  d.tower_w = at(1);
  d.head_w = at(2);
  d.bias = atf(3);
  d.qmul = atd(4);
  d.qres = atd(5);
  d.qhi = atf(6);
  d.qbias = atd(28);
  d.qext = atd(29);
  d.head_b = atf(7);
  d.fc1_w = atf(8);
  d.fc1_b = atf(9);
  d.fc2_w = atf(10);
  d.head_sc = atf(11);
  d.head_bc = atf(12);
  d.fc1_t = atf(13);
  d.fc2_b = dep ? 0.0f : v.fc2_b[0];
  if (dep) {
    d.pool_every = s.pool_every;
    d.value_channels = V;
    d.emb_w = at(14);
    d.q_w = at(15);
    d.k_w = at(16);
    d.p_w = at(17);
    d.emb_sc = atf(18);
    d.emb_bc = atf(19);
    d.q_b = atf(20);
    d.k_b = atf(21);
    d.pool_wt = atf(22);
    d.pool_m = atd(23);
    d.pool_b = atd(24);
    d.pool_cinv = atd(25);
    d.actions = reinterpret_cast<const uint32_t*>(at(26));
    d.wdl_fc1_t = atf(27);
    d.wdl_fc1_b = atf(9);
    d.wdl_fc2_w = atf(10);
    for (int i = 0; i < 3; ++i) d.wdl_fc2_b[i] = v.fc2_b[i];
  }
  *out = net;
  return AZ_OK;
}

int az_eval_batch_wdl(az_net* net, const float* planes, const uint8_t* legal, int32_t B, float* policy,
                      float* value, float* wdl, void* stream) {
  if (!net) return fail(AZ_ERR_INVALID_ARG, "NULL handle");
  if (B < 0) return fail(AZ_ERR_INVALID_ARG, "B = %d < 0", B);
  const bool dep = is_deployed(net->spec);
  if (wdl && !dep) return fail(AZ_ERR_INVALID_ARG, "wdl output needs a network with the WDL value head");
  if (B == 0) return AZ_OK;
  if (B > net->spec.max_batch) return fail(AZ_ERR_INVALID_ARG, "B = %d > max_batch %d", B, net->spec.max_batch);
  if (!planes || !legal || !policy || !value) return fail(AZ_ERR_INVALID_ARG, "NULL buffer");
  if (((uintptr_t)planes | (uintptr_t)legal | (uintptr_t)policy) & 15u)
    return fail(AZ_ERR_INVALID_ARG, "planes, legal and policy must be 16-byte aligned");
  if (((uintptr_t)value | (uintptr_t)wdl) & 3u) return fail(AZ_ERR_INVALID_ARG, "value and wdl must be 4-byte aligned");
  int cur = 0;
  hipError_t e = hipGetDevice(&cur);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (cur != net->device && (e = hipSetDevice(net->device)) != hipSuccess) return hip_fail(e, "hipSetDevice");
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (dep)
    e = (net->dtype == AZ_INT8 ? az_launch_deployed_int8 : az_launch_deployed_bf16)(
        net->dn, choose_tiling(net, B), planes, legal, B, policy, value, wdl, s);
  else if (net->dtype == AZ_F32)
    e = az_launch_f32(net->dn, planes, legal, B, policy, value, s);
  else
    e = az_launch_mfma(net->dtype, choose_tiling(net, B), net->dn, planes, legal, B, policy, value, s);
  if (cur != net->device) (void)hipSetDevice(cur);
  if (e != hipSuccess) return hip_fail(e, "kernel launch");
  return AZ_OK;
}

int az_eval_batch(az_net* net, const float* planes, const uint8_t* legal, int32_t B, float* policy,
                  float* value, void* stream) {
  return az_eval_batch_wdl(net, planes, legal, B, policy, value, nullptr, stream);
}

int az_net_moves(const az_net* net) {
  if (!net) return fail(AZ_ERR_INVALID_ARG, "NULL handle");
  return az_spec_moves(net->spec);
}

int az_net_set_tiling(az_net* net, int32_t tiling) {
  if (!net) return fail(AZ_ERR_INVALID_ARG, "NULL handle");
  const bool valid = net->dtype == AZ_F32          ? tiling == 0
                     : is_deployed(net->spec)          ? (tiling >= 0 && tiling <= 2)
                                                       : (tiling == 0 || az_mfma_tiling_valid(net->spec.filters, tiling));
  if (!valid)
    return fail(AZ_ERR_INVALID_ARG, "tiling %d not available for this dtype", tiling);
  net->tiling = tiling;
  return AZ_OK;
}

int az_net_tiling_for(const az_net* net, int32_t B) {
  if (!net) return fail(AZ_ERR_INVALID_ARG, "NULL handle");
  if (B < 0) return fail(AZ_ERR_INVALID_ARG, "B = %d < 0", B);
  return choose_tiling(net, B);
}

size_t az_net_device_bytes(const az_net* net) { return net ? net->dbytes : 0; }

void az_net_free(az_net* net) {
  if (!net) return;
  if (net->dmem) {
    int cur = 0;
    const bool have = hipGetDevice(&cur) == hipSuccess;
    if (have && cur != net->device) (void)hipSetDevice(net->device);
    az_dev_free(net->dmem);
    if (have && cur != net->device) (void)hipSetDevice(cur);
  }
  delete net;
}

}  // extern "C"
