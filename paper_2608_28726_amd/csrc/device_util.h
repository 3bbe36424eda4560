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

// Element access: a 16-byte vector holds 4 float32 or 8 bfloat16 logits.
template <typename Tin>
struct Elem;

template <>
struct Elem<float> {
  static constexpr int kVec = 4;
  __device__ __forceinline__ static void unpack(const uint4& v, float* z) {
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
  __device__ __forceinline__ static void unpack(const uint4& v, float* z) {
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

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = kWave / 2; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = kWave / 2; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

__device__ __forceinline__ double wave_sum_d(double v) {
#pragma unroll
  for (int o = kWave / 2; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

__device__ __forceinline__ uint32_t wave_sum_u(uint32_t v) {
#pragma unroll
  for (int o = kWave / 2; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
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
#pragma unroll
  for (int o = kWave / 2; o > 0; o >>= 1) {
    const float o1 = __shfl_xor(t1, o);
    const int32_t o1i = __shfl_xor(t1i, o);
    const float o2 = __shfl_xor(t2, o);
    top2_merge(t1, t1i, t2, o1, o1i, o2);
  }
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
