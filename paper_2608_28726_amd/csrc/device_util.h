// Device-side building blocks shared by the verifier kernels (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "prouter.h"

namespace pr {

constexpr int kWave = 64;
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
// Clamp for exponent arguments: any finite value this negative makes
// exp2 return 0 and keeps 0 * x finite (x = -inf would give NaN).
constexpr float kBig = 1e30f;
constexpr float kNegSentinel = -3.402823466e38f;  // -FLT_MAX: "no finite max yet"
constexpr int32_t kNoIndex = 0x7fffffff;

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Largest float strictly below x, for finite x or +inf (x == -inf has none).
__device__ __forceinline__ float next_below(float x) {
  uint32_t b = __float_as_uint(x);
  if ((b & 0x7fffffffu) == 0) return __uint_as_float(0x80000001u);  // +-0 -> -denorm_min
  return __uint_as_float((b & 0x80000000u) ? b + 1u : b - 1u);
}

// A 16-byte vector of logits as four 32-bit words. A native vector type
// keeps each load in one register quadruple, so loads carried across loop
// iterations need no register copies (which would wait for the load).
typedef uint32_t vec4u __attribute__((ext_vector_type(4)));

// Element access: a 16-byte vector holds 4 float32 or 8 bfloat16 logits.
template <typename Tin>
struct Elem;

template <>
struct Elem<float> {
  static constexpr int kVec = 4;
  __device__ __forceinline__ static void unpack(const vec4u& v, float* z) {
    z[0] = __uint_as_float(v.x);
    z[1] = __uint_as_float(v.y);
    z[2] = __uint_as_float(v.z);
    z[3] = __uint_as_float(v.w);
  }
  __device__ __forceinline__ static float load1(const void* base, int64_t i) {
    return static_cast<const float*>(base)[i];
  }
};

template <>
struct Elem<uint16_t> {  // bfloat16 bit patterns
  static constexpr int kVec = 8;
  __device__ __forceinline__ static void unpack(const vec4u& v, float* z) {
    z[0] = bf16_lo(v.x);
    z[1] = bf16_hi(v.x);
    z[2] = bf16_lo(v.y);
    z[3] = bf16_hi(v.y);
    z[4] = bf16_lo(v.z);
    z[5] = bf16_hi(v.z);
    z[6] = bf16_lo(v.w);
    z[7] = bf16_hi(v.w);
  }
  __device__ __forceinline__ static float load1(const void* base, int64_t i) {
    return __uint_as_float(static_cast<uint32_t>(static_cast<const uint16_t*>(base)[i]) << 16);
  }
};

// Reduction state of a stretch of one row. S and E are relative to the
// reference a = round(m * c) (c = log2(e) / T, the float32 product):
// S = sum 2^x, E = sum 2^x * x with x = fma(z, c, -a). References are always
// such rounded products and are compared by plain subtraction; the library is
// built with floating-point contraction off so that this stays so. t1/t1i/t2: largest value, its lowest index, second value.
// cnt: tokens of the stretch that precede the sampled token in the order.
struct Partial {
  float m;
  float S;
  float E;
  float t1;
  int32_t t1i;
  float t2;
  uint32_t cnt;
  uint32_t pad;
};

// Wave-wide reductions by DPP lane moves within the wave (no LDS round
// trips): two quad permutations, the half-row and row mirrors combine the 16
// lanes of each row, the row broadcasts of lanes 15 and 31 fold the four rows
// into lane 63, whose value every lane then reads as a scalar. Each must be
// called with all 64 lanes active.
namespace dpp {
constexpr int kXor1 = 0xB1;        // quad_perm [1,0,3,2]
constexpr int kXor2 = 0x4E;        // quad_perm [2,3,0,1]
constexpr int kHalfMirror = 0x141;  // row_half_mirror
constexpr int kMirror = 0x140;      // row_mirror
constexpr int kBcast15 = 0x142;     // row_bcast:15 (rows 1 and 3 written)
constexpr int kBcast31 = 0x143;     // row_bcast:31 (rows 2 and 3 written)

// src moved by CTRL; lanes of rows outside ROW_MASK receive `old`.
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ uint32_t mov(uint32_t old, uint32_t src) {
  return static_cast<uint32_t>(
      __builtin_amdgcn_update_dpp(static_cast<int>(old), static_cast<int>(src), CTRL, ROW_MASK, 0xf, false));
}
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ float movf(float old, float src) {
  return __uint_as_float(mov<CTRL, ROW_MASK>(__float_as_uint(old), __float_as_uint(src)));
}
template <int CTRL, int ROW_MASK>
__device__ __forceinline__ double movd(double old, double src) {
  const uint64_t o = __double_as_longlong(old), v = __double_as_longlong(src);
  const uint32_t lo = mov<CTRL, ROW_MASK>(static_cast<uint32_t>(o), static_cast<uint32_t>(v));
  const uint32_t hi = mov<CTRL, ROW_MASK>(static_cast<uint32_t>(o >> 32), static_cast<uint32_t>(v >> 32));
  return __longlong_as_double(static_cast<long long>((static_cast<uint64_t>(hi) << 32) | lo));
}
__device__ __forceinline__ float lane63(float v) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), kWave - 1));
}
__device__ __forceinline__ uint32_t lane63(uint32_t v) {
  return static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(v), kWave - 1));
}
__device__ __forceinline__ int32_t lane63(int32_t v) { return __builtin_amdgcn_readlane(v, kWave - 1); }
__device__ __forceinline__ double lane63(double v) {
  const uint64_t b = __double_as_longlong(v);
  const uint32_t lo = lane63(static_cast<uint32_t>(b)), hi = lane63(static_cast<uint32_t>(b >> 32));
  return __longlong_as_double(static_cast<long long>((static_cast<uint64_t>(hi) << 32) | lo));
}
}  // namespace dpp

__device__ __forceinline__ float wave_max(float v) {
  using namespace dpp;
  v = fmaxf(v, movf<kXor1, 0xf>(v, v));
  v = fmaxf(v, movf<kXor2, 0xf>(v, v));
  v = fmaxf(v, movf<kHalfMirror, 0xf>(v, v));
  v = fmaxf(v, movf<kMirror, 0xf>(v, v));
  v = fmaxf(v, movf<kBcast15, 0xa>(v, v));
  v = fmaxf(v, movf<kBcast31, 0xc>(v, v));
  return lane63(v);
}

__device__ __forceinline__ float wave_sum(float v) {
  using namespace dpp;
  v += movf<kXor1, 0xf>(0.0f, v);
  v += movf<kXor2, 0xf>(0.0f, v);
  v += movf<kHalfMirror, 0xf>(0.0f, v);
  v += movf<kMirror, 0xf>(0.0f, v);
  v += movf<kBcast15, 0xa>(0.0f, v);
  v += movf<kBcast31, 0xc>(0.0f, v);
  return lane63(v);
}

__device__ __forceinline__ double wave_sum_d(double v) {
  using namespace dpp;
  v += movd<kXor1, 0xf>(0.0, v);
  v += movd<kXor2, 0xf>(0.0, v);
  v += movd<kHalfMirror, 0xf>(0.0, v);
  v += movd<kMirror, 0xf>(0.0, v);
  v += movd<kBcast15, 0xa>(0.0, v);
  v += movd<kBcast31, 0xc>(0.0, v);
  return lane63(v);
}

__device__ __forceinline__ uint32_t wave_sum_u(uint32_t v) {
  using namespace dpp;
  v += mov<kXor1, 0xf>(0u, v);
  v += mov<kXor2, 0xf>(0u, v);
  v += mov<kHalfMirror, 0xf>(0u, v);
  v += mov<kMirror, 0xf>(0u, v);
  v += mov<kBcast15, 0xa>(0u, v);
  v += mov<kBcast31, 0xc>(0u, v);
  return lane63(v);
}

// (t1, t1i, t2) merge: larger value first, equal values by lower index; the
// second value is the larger of the loser's top-1 and both top-2 values.
__device__ __forceinline__ void top2_merge(float& t1, int32_t& t1i, float& t2, float o1, int32_t o1i, float o2) {
  const bool other_wins = (o1 > t1) || (o1 == t1 && o1i < t1i);
  const float loser = other_wins ? t1 : o1;
  if (other_wins) {
    t1 = o1;
    t1i = o1i;
  }
  t2 = fmaxf(fmaxf(t2, o2), loser);
}

__device__ __forceinline__ void wave_top2(float& t1, int32_t& t1i, float& t2) {
  using namespace dpp;
#define PR_TOP2I_STEP(CTRL, MASK)                                                             \
  {                                                                                           \
    const float o1 = movf<CTRL, MASK>(-INFINITY, t1);                                         \
    const int32_t o1i = static_cast<int32_t>(mov<CTRL, MASK>(static_cast<uint32_t>(kNoIndex), \
                                                             static_cast<uint32_t>(t1i)));    \
    const float o2 = movf<CTRL, MASK>(-INFINITY, t2);                                         \
    top2_merge(t1, t1i, t2, o1, o1i, o2);                                                     \
  }
  PR_TOP2I_STEP(kXor1, 0xf)
  PR_TOP2I_STEP(kXor2, 0xf)
  PR_TOP2I_STEP(kHalfMirror, 0xf)
  PR_TOP2I_STEP(kMirror, 0xf)
  PR_TOP2I_STEP(kBcast15, 0xa)
  PR_TOP2I_STEP(kBcast31, 0xc)
#undef PR_TOP2I_STEP
  t1 = dpp::lane63(t1);
  t1i = dpp::lane63(t1i);
  t2 = dpp::lane63(t2);
}

// Rescale factor from a stretch's reference a_l to the row reference A.
// A stretch that saw no finite logit contributes nothing (but NaN sums stay
// NaN); its reference may be a sentinel while A is -inf, so no exponent is
// formed for it.
__device__ __forceinline__ void rebase(bool no_finite, float a_l, float A, float& S, float& E) {
  if (no_finite) {
    S *= 0.0f;
    E *= 0.0f;
    return;
  }
  const float d = fmaxf(a_l - A, -kBig);
  const float s = fast_exp2(d);
  E = s * E + (s * d) * S;
  S = s * S;
}

// ln S of a row's sum of exps relative to its largest logit (S >= 1: that
// logit contributes 1). Below 2, S - 1 is exact (Sterbenz) and log1p keeps
// the relative precision of the small logarithm of an almost one-hot row.
__device__ __forceinline__ float ln_sum(float S) { return S < 2.0f ? log1pf(S - 1.0f) : logf(S); }
__device__ __forceinline__ double ln_sum(double S) { return S < 2.0 ? log1p(S - 1.0) : log(S); }

// Smallest accepted temperature: keeps log2(e) / T finite in float32.
constexpr float kMinTemperature = 0x1p-100f;

// A temperature the path accepts: finite and at least 2^-100.
__device__ __forceinline__ bool temperature_ok(float T) { return T >= kMinTemperature && T < INFINITY; }

// Sortable 32-bit key of a float: unsigned order equals numeric order,
// -0 maps to +0, NaN sorts above +inf.
__device__ __forceinline__ uint32_t float_key(float f) {
  uint32_t b = __float_as_uint(f);
  if (b == 0x80000000u) b = 0u;
  return (b & 0x80000000u) ? ~b : (b | 0x80000000u);
}
__device__ __forceinline__ float key_float(uint32_t k) {
  return __uint_as_float((k & 0x80000000u) ? (k & 0x7fffffffu) : ~k);
}

}  // namespace pr
