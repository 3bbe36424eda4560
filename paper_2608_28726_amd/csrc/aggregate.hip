// Per-request summaries, score and ship rule (Pro-Router, Sec. 3.1: the
// stacked per-token feature sequence of a request, one shipping confidence,
// ship iff p >= tau; Sec. 4.2, Table "ablation": a quantile summary of the
// sequence as verifier input).
//
// One workgroup per request. For each confidence column
// A = (logprob, maxprob, -entropy, margin) it computes the count, the mean
// (double sums), the minimum and the exact nearest-rank q-quantile by a
// four-pass byte-wise radix select over order-preserving 32-bit keys, with
// a 256-bin histogram in LDS. The same code serves the offline ragged batch
// (segments given by offsets) and the streaming state (each slot's history).
#include "aggregate.h"

namespace pr {

namespace {

constexpr int kAggBlock = 256;

struct AggOut {
  double mean_d;  // unrounded mean, used by the score
  float mean, min, quant;
};

// Confidence column f of row r of the per-token feature arrays.
struct FeatCol {
  const float* p;
  bool negate;
  __device__ __forceinline__ float operator()(int64_t r) const { return negate ? -p[r] : p[r]; }
};

struct HistCol {
  const float* p;
  __device__ __forceinline__ float operator()(int64_t r) const { return p[r]; }
};

// Block-wide summaries of n values get(lo + i). All threads return the result.
template <int BLOCK, typename Get>
__device__ AggOut block_summaries(Get get, int64_t lo, int64_t n, int64_t j, bool quant_ok) {
  constexpr int NW = BLOCK / kWave;
  __shared__ double sh_sum[NW];
  __shared__ float sh_min[NW];
  __shared__ uint32_t sh_nan[NW];
  __shared__ uint32_t hist[256];
  __shared__ uint32_t sh_prefix, sh_j;
  const int t = threadIdx.x;
  const int lane = t % kWave, w = t / kWave;
  const float qnan = __uint_as_float(0x7fc00000u);

  double s = 0.0;
  float mn = INFINITY;
  uint32_t has_nan = 0;
  for (int64_t i = t; i < n; i += BLOCK) {
    const float v = get(lo + i);
    if (v != v) {
      has_nan = 1;
    } else {
      s += static_cast<double>(v);
      mn = fminf(mn, v);
    }
  }
  s = wave_sum_d(s);
  mn = -wave_max(-mn);
  has_nan = wave_sum_u(has_nan);
  if (lane == 0) {
    sh_sum[w] = s;
    sh_min[w] = mn;
    sh_nan[w] = has_nan;
  }
  __syncthreads();
  double tot = 0.0;
  float gmin = INFINITY;
  uint32_t nan_any = 0;
  for (int k = 0; k < NW; ++k) {
    tot += sh_sum[k];
    gmin = fminf(gmin, sh_min[k]);
    nan_any |= sh_nan[k];
  }
  AggOut o;
  if (n == 0 || nan_any) {
    o.mean = o.min = o.quant = qnan;
    o.mean_d = static_cast<double>(qnan);
    __syncthreads();
    return o;
  }
  o.mean_d = tot / static_cast<double>(n);
  o.mean = static_cast<float>(o.mean_d);
  o.min = gmin;
  if (!quant_ok) {
    o.quant = qnan;
    __syncthreads();
    return o;
  }

  // Radix select of the j-th smallest key, most significant byte first.
  uint32_t prefix = 0, mask = 0;
  if (t == 0) sh_j = static_cast<uint32_t>(j);
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 24 - 8 * pass;
    for (int b = t; b < 256; b += BLOCK) hist[b] = 0;
    __syncthreads();
    for (int64_t i = t; i < n; i += BLOCK) {
      const uint32_t k = float_key(get(lo + i));
      if ((k & mask) == prefix) atomicAdd(&hist[(k >> shift) & 255u], 1u);
    }
    __syncthreads();
    if (t == 0) {
      uint32_t need = sh_j, b = 0;
      for (; b < 255; ++b) {
        if (need <= hist[b]) break;
        need -= hist[b];
      }
      sh_j = need;
      sh_prefix = prefix | (b << shift);
    }
    __syncthreads();
    prefix = sh_prefix;
    mask |= 255u << shift;
    __syncthreads();
  }
  o.quant = key_float(prefix);
  return o;
}

__device__ int64_t quant_rank(double q, int64_t n) {
  double qn = q * static_cast<double>(n);
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

}  // namespace

__global__ __launch_bounds__(kAggBlock) void aggregate_kernel(pr_token_features_t feats, const int32_t* offsets,
                                                              int32_t n_req, AggParamsDev hp,
                                                              pr_request_agg_t out) {
  const int64_t i = blockIdx.x;
  if (i >= n_req) return;
  const int64_t lo = offsets[i];
  const int64_t hi = offsets[i + 1];
  const int64_t n = hi > lo ? hi - lo : 0;
  const int64_t j = n > 0 ? quant_rank(hp.q, n) : 1;
  const float* cols[4] = {feats.logprob, feats.maxprob, feats.entropy, feats.margin};
  float mean[4], mn[4], qu[4];
  double mean_d[4];
  for (int f = 0; f < 4; ++f) {
    const FeatCol get{cols[f], f == 2};
    const AggOut o = block_summaries<kAggBlock>(get, lo, n, j, true);
    mean[f] = o.mean;
    mn[f] = o.min;
    qu[f] = o.quant;
    mean_d[f] = o.mean_d;
    __syncthreads();
  }
  if (threadIdx.x == 0) write_request(out, i, n, mean, mn, qu, head_score(hp, mean_d, mn, qu, n));
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
  }
}

// One workgroup per finishing slot: summaries as in aggregate_kernel, with
// the running sums and minima taken from the slot state and the quantile
// selected from the slot's history; then the slot is cleared.
__global__ __launch_bounds__(kAggBlock) void stream_finish_kernel(StreamDev s, const int32_t* slots, int32_t n,
                                                                  AggParamsDev hp, float thr,
                                                                  pr_request_agg_t out, uint8_t* ship) {
  const int64_t i = blockIdx.x;
  if (i >= n) return;
  const int32_t slot = slots[i];
  const bool ok = slot >= 0 && slot < s.max_slots;
  const int64_t cnt = ok ? s.count[slot] : 0;
  const float qnan = __uint_as_float(0x7fc00000u);
  float mean[4], mn[4], qu[4];
  double mean_d[4];
  const int64_t j = cnt > 0 ? quant_rank(hp.q, cnt) : 1;
  const bool kept = cnt <= s.max_len;
  for (int f = 0; f < 4; ++f) {
    const bool bad = cnt == 0 || (ok && ((s.nanbits[slot] >> f) & 1u));
    if (bad) {
      mean[f] = mn[f] = qu[f] = qnan;
      mean_d[f] = static_cast<double>(qnan);
      continue;
    }
    mean_d[f] = s.sum[slot * 4 + f] / static_cast<double>(cnt);
    mean[f] = static_cast<float>(mean_d[f]);
    mn[f] = s.minv[slot * 4 + f];
    if (kept) {
      const HistCol get{s.hist + (static_cast<int64_t>(slot) * 4 + f) * s.max_len};
      qu[f] = block_summaries<kAggBlock>(get, 0, cnt, j, true).quant;
    } else {
      qu[f] = qnan;
    }
    __syncthreads();
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    const float score = head_score(hp, mean_d, mn, qu, cnt);
    write_request(out, i, cnt, mean, mn, qu, score);
    if (ship) ship[i] = score >= thr ? 1 : 0;
    if (ok) {
      s.count[slot] = 0;
      s.nanbits[slot] = 0;
      for (int f = 0; f < 4; ++f) {
        s.sum[slot * 4 + f] = 0.0;
        s.minv[slot * 4 + f] = INFINITY;
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
