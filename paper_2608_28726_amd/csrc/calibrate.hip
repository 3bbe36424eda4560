// Threshold calibration for a ship fraction (Pro-Router, Sec. 3.1: the ship
// rule p >= tau with tau fixed in advance on a validation pool; Sec. 4.1: the
// coverage rule of selective prediction, a ship fraction q).
//
// tau is the k-th largest non-NaN score of the pool, k = max(1, ceil(q n))
// over the n non-NaN scores, and n_ship = #{s >= tau}. One workgroup of 1024
// threads: a count of the non-NaN scores, then a byte-wise radix select of
// the (n - k + 1)-th smallest order-preserving key (four passes, each a
// 256-bin LDS histogram per wave summed over the waves and scanned by one
// wave). The select also yields the position of tau among the scores equal
// to it, which gives n_ship without another pass. Pools of up to 16,384
// scores are read once into registers; larger ones are re-read on each pass
// (from L2).
#include "calibrate.h"

namespace pr {

namespace {

constexpr int kCalBlock = 1024;
constexpr int kCalWaves = kCalBlock / kWave;
constexpr int kCalRegKeys = 16;

// Key of a score: numeric order, -0 == +0, NaN above everything (it is
// never selected: the rank asked for is at most the number of non-NaN
// scores).
__device__ __forceinline__ uint32_t score_key(float v) {
  return v != v ? 0xffffffffu : float_key(v);
}

struct CalShared {
  uint32_t hist[kCalWaves][256];
  uint32_t tot[256];
  uint32_t wsum[kCalWaves];
  uint32_t sel[2];
};

// Adds the key's digit to this wave's histogram; a wave whose active lanes
// all share one digit adds once (pools of confidences crowd into few bins).
__device__ __forceinline__ void hist_add(uint32_t* h, uint32_t digit) {
  const uint32_t first = __builtin_amdgcn_readfirstlane(digit);
  const uint64_t active = __ballot(1);
  const uint64_t same = __ballot(digit == first);
  if (same == active) {
    if ((threadIdx.x % kWave) == static_cast<unsigned>(__builtin_ctzll(active)))
      atomicAdd(&h[first], static_cast<uint32_t>(__popcll(active)));
  } else {
    atomicAdd(&h[digit], 1u);
  }
}

template <bool REG>
__device__ void calibrate_body(const float* scores, int32_t n, double q, float* tau, int32_t* n_ship,
                               CalShared& sh) {
  const int t = threadIdx.x;
  const int w = t / kWave;
  const int lane = t % kWave;
  uint32_t keys[REG ? kCalRegKeys : 1];
  uint32_t valid = 0;
  if constexpr (REG) {
#pragma unroll
    for (int r = 0; r < kCalRegKeys; ++r) {
      const int64_t i = t + static_cast<int64_t>(r) * kCalBlock;
      const float v = i < n ? scores[i] : __uint_as_float(0x7fc00000u);
      keys[r] = score_key(v);
      valid += keys[r] != 0xffffffffu ? 1u : 0u;
    }
  } else {
    for (int64_t i = t; i < n; i += kCalBlock) valid += scores[i] == scores[i] ? 1u : 0u;
  }
  valid = wave_sum_u(valid);
  if (lane == 0) sh.wsum[w] = valid;
  __syncthreads();
  uint32_t nv = 0;
#pragma unroll
  for (int k = 0; k < kCalWaves; ++k) nv += sh.wsum[k];
  if (q == 0.0 || nv == 0) {
    if (t == 0) {
      tau[0] = INFINITY;
      if (n_ship) n_ship[0] = 0;
    }
    return;
  }
  int64_t k = static_cast<int64_t>(ceil(q * static_cast<double>(nv)));
  if (k < 1) k = 1;
  if (k > nv) k = nv;
  const uint32_t j = nv - static_cast<uint32_t>(k) + 1;  // j-th smallest
  uint32_t prefix = 0, mask = 0, need = j;
  uint32_t* h = sh.hist[w];
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    for (int b = lane; b < 256; b += kWave) h[b] = 0;
    __syncthreads();
    if constexpr (REG) {
#pragma unroll
      for (int r = 0; r < kCalRegKeys; ++r)
        if ((keys[r] & mask) == prefix) hist_add(h, (keys[r] >> shift) & 255u);
    } else {
      for (int64_t i = t; i < n; i += kCalBlock) {
        const uint32_t key = score_key(scores[i]);
        if ((key & mask) == prefix) hist_add(h, (key >> shift) & 255u);
      }
    }
    __syncthreads();
    if (t < 256) {
      uint32_t c = 0;
#pragma unroll
      for (int v = 0; v < kCalWaves; ++v) c += sh.hist[v][t];
      sh.tot[t] = c;
    }
    __syncthreads();
    if (w == 0) {
      const uint32_t c0 = sh.tot[4 * lane], c1 = sh.tot[4 * lane + 1], c2 = sh.tot[4 * lane + 2],
                     c3 = sh.tot[4 * lane + 3];
      const uint32_t cnt = c0 + c1 + c2 + c3;
      uint32_t incl = cnt;
#pragma unroll
      for (int o = 1; o < kWave; o <<= 1) {
        const uint32_t u = __shfl_up(incl, o);
        if (lane >= o) incl += u;
      }
      const uint32_t excl = incl - cnt;
      if (need > excl && need <= incl) {
        uint32_t r = need - excl, b = 0;
        if (r > c0) {
          r -= c0;
          b = 1;
          if (r > c1) {
            r -= c1;
            b = 2;
            if (r > c2) {
              r -= c2;
              b = 3;
            }
          }
        }
        sh.sel[0] = 4u * lane + b;
        sh.sel[1] = r;
      }
    }
    __syncthreads();
    prefix |= sh.sel[0] << shift;
    need = sh.sel[1];
    mask |= 255u << shift;
    __syncthreads();  // sel is rewritten by the next pass
  }
  if (t == 0) {
    // The j-th smallest is the need-th of the scores equal to tau: j - need
    // scores lie below it, every other non-NaN score ships.
    tau[0] = key_float(prefix);
    if (n_ship) n_ship[0] = static_cast<int32_t>(nv - (j - need));
  }
}

__global__ __launch_bounds__(kCalBlock) void calibrate_kernel(const float* scores, int32_t n, double q, float* tau,
                                                              int32_t* n_ship) {
  __shared__ CalShared sh;
  if (n <= kCalRegKeys * kCalBlock)
    calibrate_body<true>(scores, n, q, tau, n_ship, sh);
  else
    calibrate_body<false>(scores, n, q, tau, n_ship, sh);
}

}  // namespace

hipError_t launch_calibrate(const float* scores, int32_t n, double q, float* tau, int32_t* n_ship,
                            hipStream_t stream) {
  calibrate_kernel<<<1, kCalBlock, 0, stream>>>(scores, n, q, tau, n_ship);
  return hipGetLastError();
}

}  // namespace pr
