// Per-request summaries, score and ship rule (Pro-Router, Sec. 3.1: the
// stacked per-token feature sequence of a request, one shipping confidence,
// ship iff p >= tau; Sec. 4.2, Table "ablation": a quantile summary of the
// sequence as verifier input).
//
// One workgroup per request, one wave per confidence column
// A = (logprob, maxprob, -entropy, margin): count, mean (double sums),
// minimum and the exact nearest-rank q-quantile by a four-pass byte-wise radix
// select over order-preserving 32-bit keys (a 256-bin LDS histogram per wave
// and a wave prefix scan per pass). The same code serves the offline ragged
// batch (segments given by offsets) and the streaming state (each slot's
// history).
#include "aggregate.h"
#include "p2.h"

namespace pr {

namespace {

// Four waves per workgroup: wave f summarises confidence column f.
constexpr int kAggBlock = 4 * kWave;

// Confidence column of the per-token feature arrays (entropy is negated).
struct FeatCol {
  const float* p;
  bool negate;
  __device__ __forceinline__ float operator()(int64_t r) const { return negate ? -p[r] : p[r]; }
};

struct HistCol {
  const float* p;
  __device__ __forceinline__ float operator()(int64_t r) const { return p[r]; }
};

__device__ __forceinline__ uint32_t wave_incl_scan_u(uint32_t v, int lane) {
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const uint32_t t = __shfl_up(v, o);
    if (lane >= o) v += t;
  }
  return v;
}

// Sum (double), minimum and NaN presence of the wave's n values get(lo + k).
template <typename Get>
__device__ void wave_stats(Get get, int64_t lo, int64_t n, double& sum, float& mn, bool& has_nan) {
  const int lane = threadIdx.x % kWave;
  double s = 0.0;
  float m = INFINITY;
  uint32_t nan = 0;
  for (int64_t k = lane; k < n; k += kWave) {
    const float v = get(lo + k);
    if (v != v) {
      nan = 1;
    } else {
      s += static_cast<double>(v);
      m = fminf(m, v);
    }
  }
  sum = wave_sum_d(s);
  mn = -wave_max(-m);
  has_nan = wave_sum_u(nan) != 0;
}

// Byte-wise radix select of the j-th smallest (1-based) key: per pass a
// 256-bin histogram of the keys that match the digits chosen so far, then a
// wave prefix scan locates the bin holding the j-th key. Every wave of the
// block must call this with the same n (it uses block barriers).
// hist: [4][256], sel: [4][2] in LDS. keys(k) yields the k-th key.
template <typename Keys>
__device__ uint32_t radix_select_keys(Keys keys, int64_t n, int64_t j, uint32_t* hist, uint32_t* sel) {
  const int w = threadIdx.x / kWave;
  const int lane = threadIdx.x % kWave;
  uint32_t* h = hist + w * 256;
  uint32_t prefix = 0, mask = 0, need = static_cast<uint32_t>(j);
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    for (int b = lane; b < 256; b += kWave) h[b] = 0;
    __syncthreads();
    keys.for_each([&](uint32_t key) {
      if ((key & mask) == prefix) atomicAdd(&h[(key >> shift) & 255u], 1u);
    });
    __syncthreads();
    const uint32_t c0 = h[4 * lane], c1 = h[4 * lane + 1], c2 = h[4 * lane + 2], c3 = h[4 * lane + 3];
    const uint32_t tot = c0 + c1 + c2 + c3;
    const uint32_t incl = wave_incl_scan_u(tot, lane);
    const uint32_t excl = incl - tot;
    if (need > excl && need <= incl) {
      uint32_t r = need - excl, q = 0;
      if (r > c0) {
        r -= c0;
        q = 1;
        if (r > c1) {
          r -= c1;
          q = 2;
          if (r > c2) {
            r -= c2;
            q = 3;
          }
        }
      }
      sel[2 * w] = 4u * lane + q;
      sel[2 * w + 1] = r;
    }
    __syncthreads();
    prefix |= sel[2 * w] << shift;
    need = sel[2 * w + 1];
    mask |= 255u << shift;
  }
  return prefix;
}

// Keys read from memory on every pass (any n).
template <typename Get>
struct MemKeys {
  Get get;
  int64_t lo, n;
  template <typename Fn>
  __device__ __forceinline__ void for_each(Fn fn) const {
    for (int64_t k = threadIdx.x % kWave; k < n; k += kWave) fn(float_key(get(lo + k)));
  }
};

// Keys held in registers, R per lane (n <= R * 64): one read for all passes.
template <int R>
struct RegKeys {
  uint32_t k[R];
  int cnt;  // keys this lane holds
  template <typename Fn>
  __device__ __forceinline__ void for_each(Fn fn) const {
#pragma unroll
    for (int r = 0; r < R; ++r)
      if (r < cnt) fn(k[r]);
  }
};

constexpr int kRegKeys = 16;  // up to 1,024 values per column stay in registers

// The j-th smallest of the wave's n values get(lo + k).
template <typename Get>
__device__ float radix_select(Get get, int64_t lo, int64_t n, int64_t j, uint32_t* hist, uint32_t* sel) {
  if (n <= static_cast<int64_t>(kRegKeys) * kWave) {
    RegKeys<kRegKeys> rk;
    rk.cnt = 0;
    const int lane = threadIdx.x % kWave;
#pragma unroll
    for (int r = 0; r < kRegKeys; ++r) {
      const int64_t k = lane + static_cast<int64_t>(r) * kWave;
      rk.k[r] = k < n ? float_key(get(lo + k)) : 0u;
      rk.cnt += k < n ? 1 : 0;
    }
    return key_float(radix_select_keys(rk, n, j, hist, sel));
  }
  return key_float(radix_select_keys(MemKeys<Get>{get, lo, n}, n, j, hist, sel));
}

// Sum (double), minimum, NaN presence and the j-th smallest of the wave's n
// values get(lo + k): up to kRegKeys per lane they are read once and both
// the statistics and the select work from registers (the sums in the order
// of wave_stats), more are read by each.
template <typename Get>
__device__ float column_summary(Get get, int64_t lo, int64_t n, int64_t j, uint32_t* hist, uint32_t* sel,
                                double& sum, float& mn, bool& has_nan) {
  if (n > static_cast<int64_t>(kRegKeys) * kWave) {
    wave_stats(get, lo, n, sum, mn, has_nan);
    return key_float(radix_select_keys(MemKeys<Get>{get, lo, n}, n, j, hist, sel));
  }
  const int lane = threadIdx.x % kWave;
  float v[kRegKeys];
#pragma unroll
  for (int r = 0; r < kRegKeys; ++r) {
    const int64_t k = lane + static_cast<int64_t>(r) * kWave;
    v[r] = k < n ? get(lo + k) : 0.0f;
  }
  double s = 0.0;
  float m = INFINITY;
  uint32_t nan = 0;
  RegKeys<kRegKeys> rk;
  rk.cnt = 0;
#pragma unroll
  for (int r = 0; r < kRegKeys; ++r) {
    const bool in = lane + static_cast<int64_t>(r) * kWave < n;
    if (in) {
      if (v[r] != v[r]) {
        nan = 1;
      } else {
        s += static_cast<double>(v[r]);
        m = fminf(m, v[r]);
      }
    }
    rk.k[r] = in ? float_key(v[r]) : 0u;
    rk.cnt += in ? 1 : 0;
  }
  sum = wave_sum_d(s);
  mn = -wave_max(-m);
  has_nan = wave_sum_u(nan) != 0;
  return n > 0 ? key_float(radix_select_keys(rk, n, j, hist, sel)) : 0.0f;
}

__device__ int64_t quant_rank(double q, int64_t n) {
  const double qn = q * static_cast<double>(n);
  int64_t j = static_cast<int64_t>(ceil(qn));
  if (j < 1) j = 1;
  if (j > n) j = n;
  return j;
}

__device__ float head_score(const AggParamsDev& hp, const double* mean_d, const float* mn, const float* qu,
                            int64_t n) {
  if (n == 0) return __uint_as_float(0x7fc00000u);
  double s = hp.b;
  for (int f = 0; f < 4; ++f) {
    if (hp.w[f] != 0.0) s += hp.w[f] * mean_d[f];
    if (hp.w[4 + f] != 0.0) s += hp.w[4 + f] * static_cast<double>(mn[f]);
    if (hp.w[8 + f] != 0.0) s += hp.w[8 + f] * static_cast<double>(qu[f]);
  }
  if (hp.link == 1) s = 1.0 / (1.0 + exp(-s));
  return static_cast<float>(s);
}

__device__ void write_request(const pr_request_agg_t& out, int64_t i, int64_t n, const float* mean,
                              const float* mn, const float* qu, float score) {
  if (out.count) out.count[i] = static_cast<int32_t>(n);
  for (int f = 0; f < 4; ++f) {
    if (out.mean) out.mean[i * 4 + f] = mean[f];
    if (out.min) out.min[i * 4 + f] = mn[f];
    if (out.quant) out.quant[i * 4 + f] = qu[f];
  }
  if (out.score) out.score[i] = score;
}

struct AggShared {
  uint32_t hist[4 * 256];
  uint32_t sel[8];
  double mean_d[4];
  float mn[4], qu[4];
  uint32_t nan[4];
};

// Thread 0: applies the NaN / empty rules and writes one request.
__device__ void finish_request(const AggShared& sh, const AggParamsDev& hp, const pr_request_agg_t& out, int64_t i,
                               int64_t n, float* score_out) {
  const float qnan = __uint_as_float(0x7fc00000u);
  float mean[4], mn[4], qu[4];
  double mean_d[4];
  for (int f = 0; f < 4; ++f) {
    const bool bad = n == 0 || sh.nan[f];
    mean_d[f] = bad ? static_cast<double>(qnan) : sh.mean_d[f];
    mean[f] = bad ? qnan : static_cast<float>(sh.mean_d[f]);
    mn[f] = bad ? qnan : sh.mn[f];
    qu[f] = bad ? qnan : sh.qu[f];
  }
  const float score = head_score(hp, mean_d, mn, qu, n);
  write_request(out, i, n, mean, mn, qu, score);
  *score_out = score;
}

}  // namespace

__global__ __launch_bounds__(kAggBlock) void aggregate_kernel(pr_token_features_t feats, const int32_t* offsets,
                                                              int32_t n_req, AggParamsDev hp,
                                                              pr_request_agg_t out) {
  __shared__ AggShared sh;
  const int64_t i = blockIdx.x;
  if (i >= n_req) return;
  const int64_t lo = offsets[i];
  const int64_t hi = offsets[i + 1];
  const int64_t n = hi > lo ? hi - lo : 0;
  const int w = threadIdx.x / kWave;
  const float* cols[4] = {feats.logprob, feats.maxprob, feats.entropy, feats.margin};
  const FeatCol get{cols[w], w == 2};
  double sum;
  float mn;
  bool nan;
  const float q = column_summary(get, lo, n, n > 0 ? quant_rank(hp.q, n) : 1, sh.hist, sh.sel, sum, mn, nan);
  if (threadIdx.x % kWave == 0) {
    sh.mean_d[w] = n > 0 ? sum / static_cast<double>(n) : 0.0;
    sh.mn[w] = mn;
    sh.qu[w] = q;
    sh.nan[w] = nan ? 1u : 0u;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float score;
    finish_request(sh, hp, out, i, n, &score);
  }
}

__global__ __launch_bounds__(1024) void route_kernel(const float* scores, int32_t n_req, float thr, uint8_t* ship,
                                                     int32_t* n_ship) {
  __shared__ uint32_t sh[1024 / kWave];
  uint32_t cnt = 0;
  for (int64_t i = threadIdx.x; i < n_req; i += blockDim.x) {
    const uint8_t s = scores[i] >= thr ? 1 : 0;  // NaN compares false: escalate
    ship[i] = s;
    cnt += s;
  }
  cnt = wave_sum_u(cnt);
  if (threadIdx.x % kWave == 0) sh[threadIdx.x / kWave] = cnt;
  __syncthreads();
  if (threadIdx.x == 0 && n_ship) {
    uint32_t tot = 0;
    for (int k = 0; k < static_cast<int>(blockDim.x / kWave); ++k) tot += sh[k];
    n_ship[0] = static_cast<int32_t>(tot);
  }
}

__global__ void stream_clear_kernel(StreamDev s, const int32_t* slots, int32_t n) {
  const int64_t k = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t total = slots ? n : s.max_slots;
  if (k >= total) return;
  const int32_t slot = slots ? slots[k] : static_cast<int32_t>(k);
  if (slot < 0 || slot >= s.max_slots) return;
  s.count[slot] = 0;
  s.nanbits[slot] = 0;
  for (int f = 0; f < 4; ++f) {
    s.sum[slot * 4 + f] = 0.0;
    s.minv[slot * 4 + f] = INFINITY;
    if (s.p2q) p2::positions(s, slot, f)[12] = 0;
  }
}

// One workgroup per finishing slot: the running sums and minima come from the
// slot state, the quantile is selected from the slot's history (wave f: column
// f), or read from its P-square markers in bounded-memory mode; then the slot
// is cleared.
__global__ __launch_bounds__(kAggBlock) void stream_finish_kernel(StreamDev s, const int32_t* slots, int32_t n,
                                                                  AggParamsDev hp, float thr,
                                                                  pr_request_agg_t out, uint8_t* ship) {
  __shared__ AggShared sh;
  const int64_t i = blockIdx.x;
  if (i >= n) return;
  const int32_t slot = slots[i];
  const bool ok = slot >= 0 && slot < s.max_slots;
  const int64_t cnt = ok ? s.count[slot] : 0;
  const bool kept = cnt <= s.max_len;
  const int w = threadIdx.x / kWave;
  // The slot's running sums, minima and NaN bits are read before the
  // quantile select, so that their latency overlaps the history's.
  double sum = 0.0;
  float mn = 0.0f;
  uint32_t nanb = 0;
  if (cnt > 0) {
    sum = s.sum[slot * 4 + w];
    mn = s.minv[slot * 4 + w];
    nanb = s.nanbits[slot];
  }
  float q = __uint_as_float(0x7fc00000u);
  if (s.p2q) {
    if (cnt > 0) q = p2::estimate(s, slot, w);
  } else if (cnt > 0 && kept) {
    const HistCol get{s.hist + (static_cast<int64_t>(slot) * 4 + w) * s.max_len};
    q = radix_select(get, 0, cnt, quant_rank(hp.q, cnt), sh.hist, sh.sel);
  }
  if (threadIdx.x % kWave == 0) {
    sh.mean_d[w] = cnt > 0 ? sum / static_cast<double>(cnt) : 0.0;
    sh.mn[w] = mn;
    sh.qu[w] = q;
    sh.nan[w] = ((nanb >> w) & 1u) ? 1u : 0u;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float score;
    finish_request(sh, hp, out, i, cnt, &score);
    if (ship) ship[i] = score >= thr ? 1 : 0;
    if (ok) {
      s.count[slot] = 0;
      s.nanbits[slot] = 0;
      for (int f = 0; f < 4; ++f) {
        s.sum[slot * 4 + f] = 0.0;
        s.minv[slot * 4 + f] = INFINITY;
        if (s.p2q) p2::positions(s, slot, f)[12] = 0;
      }
    }
  }
}

hipError_t launch_aggregate(const pr_token_features_t& feats, const int32_t* offsets, int32_t n_req,
                            const AggParamsDev& hp, const pr_request_agg_t& out, hipStream_t stream) {
  if (n_req == 0) return hipSuccess;
  aggregate_kernel<<<dim3(static_cast<unsigned>(n_req)), kAggBlock, 0, stream>>>(feats, offsets, n_req, hp, out);
  return hipGetLastError();
}

hipError_t launch_route(const float* scores, int32_t n_req, float thr, uint8_t* ship, int32_t* n_ship,
                        hipStream_t stream) {
  route_kernel<<<1, 1024, 0, stream>>>(scores, n_req, thr, ship, n_ship);
  return hipGetLastError();
}

hipError_t launch_stream_clear(const StreamDev& s, const int32_t* slots, int32_t n, hipStream_t stream) {
  const int64_t total = slots ? n : s.max_slots;
  if (total == 0) return hipSuccess;
  const unsigned blocks = static_cast<unsigned>((total + 255) / 256);
  stream_clear_kernel<<<blocks, 256, 0, stream>>>(s, slots, n);
  return hipGetLastError();
}

hipError_t launch_stream_finish(const StreamDev& s, const int32_t* slots, int32_t n, const AggParamsDev& hp,
                                float thr, const pr_request_agg_t& out, uint8_t* ship, hipStream_t stream) {
  if (n == 0) return hipSuccess;
  stream_finish_kernel<<<dim3(static_cast<unsigned>(n)), kAggBlock, 0, stream>>>(s, slots, n, hp, thr, out, ship);
  return hipGetLastError();
}

}  // namespace pr
