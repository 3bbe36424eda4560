// Threshold calibration for a ship fraction (Pro-Router, Sec. 3.1: the ship
// rule p >= tau with tau fixed in advance on a validation pool; Sec. 4.1: the
// coverage rule of selective prediction, a ship fraction q).
//
// tau is the k-th largest non-NaN score of the pool, k = max(1, ceil(q n))
// over the n non-NaN scores, and n_ship = #{s >= tau}. The select looks for
// the (n - k + 1)-th smallest order-preserving key:
//  - a range pass counts the non-NaN scores and finds their smallest and
//    largest key; the leading bits all keys share follow from these two and
//    are skipped (a pool of confidences in [0.25, 1) shares its leading seven
//    bits, which would otherwise send every score into two bins);
//  - each following pass histograms the next 11 bits of the keys that match
//    the digits chosen so far (2,048 bins), and a block-wide scan locates the
//    bin holding the wanted rank: at most three passes.
// The select also yields the position of tau among the scores equal to it,
// which gives n_ship without another pass.
//
// Pools of up to 16,384 scores run in one workgroup of 1,024 threads, the
// keys held in registers (16 per thread). Larger pools are spread over up to
// 256 workgroups per pass: a range kernel, a one-workgroup init kernel, then
// per pass a histogram kernel (LDS histogram per workgroup, its non-zero bins
// added to a global histogram) and a one-workgroup select kernel, the state
// between them in the caller's workspace.
#include "calibrate.h"

namespace pr {

namespace {

constexpr int kCalBlock = 1024;
constexpr int kCalWaves = kCalBlock / kWave;
constexpr int kCalRegKeys = 16;
constexpr int kDigit = 11;
constexpr int kBins = 1 << kDigit;
constexpr uint32_t kNanKey = 0xffffffffu;

// Key of a score: numeric order, -0 == +0, NaN above everything (it is
// never selected: the rank asked for is at most the number of non-NaN
// scores, and NaN keys are left out of the range reduction).
__device__ __forceinline__ uint32_t score_key(float v) { return v != v ? kNanKey : float_key(v); }

struct CalShared {
  uint32_t hist[kBins];
  uint32_t wcnt[kCalWaves];
  uint32_t wmin[kCalWaves];
  uint32_t wmax[kCalWaves];
  uint32_t sel[2];
};

__device__ __forceinline__ uint32_t wave_min_u(uint32_t v) {
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) v = min(v, static_cast<uint32_t>(__shfl_xor(v, o)));
  return v;
}
__device__ __forceinline__ uint32_t wave_max_u(uint32_t v) {
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) v = max(v, static_cast<uint32_t>(__shfl_xor(v, o)));
  return v;
}

// Adds one to the digit's bin; a wave whose active lanes all share one digit
// adds once.
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

// The select's progress: the digits chosen so far (prefix under mask), the
// bits still to resolve (above bit 0, below `pos`) and the rank among the
// keys that match.
struct Select {
  uint32_t nv;      // non-NaN scores
  uint32_t j;       // rank of tau among them, from the smallest
  uint32_t prefix;
  uint32_t mask;
  uint32_t need;
  int32_t pos;      // 0: done (tau and n_ship written)
};

// Block-wide combination of each thread's count and key range (threads with
// nothing to add pass 0, ~0u, 0).
__device__ void block_range(uint32_t valid, uint32_t kmin, uint32_t kmax, CalShared& sh, uint32_t& nv,
                            uint32_t& lo, uint32_t& hi) {
  const int w = threadIdx.x / kWave;
  valid = wave_sum_u(valid);
  kmin = wave_min_u(kmin);
  kmax = wave_max_u(kmax);
  if (threadIdx.x % kWave == 0) {
    sh.wcnt[w] = valid;
    sh.wmin[w] = kmin;
    sh.wmax[w] = kmax;
  }
  __syncthreads();
  nv = 0;
  lo = 0xffffffffu;
  hi = 0;
#pragma unroll
  for (int v = 0; v < kCalWaves; ++v) {
    nv += sh.wcnt[v];
    lo = min(lo, sh.wmin[v]);
    hi = max(hi, sh.wmax[v]);
  }
}

// The select's start from the pool's count and key range; writes tau and
// n_ship at once (pos = 0) when nothing ships or every score is equal.
__device__ Select select_start(uint32_t nv, uint32_t kmin, uint32_t kmax, double q, float* tau,
                               int32_t* n_ship) {
  Select s{};
  s.nv = nv;
  if (q == 0.0 || nv == 0) {
    if (threadIdx.x == 0) {
      tau[0] = INFINITY;
      if (n_ship) n_ship[0] = 0;
    }
    s.pos = 0;
    return s;
  }
  int64_t k = static_cast<int64_t>(ceil(q * static_cast<double>(nv)));
  if (k < 1) k = 1;
  if (k > nv) k = nv;
  s.j = nv - static_cast<uint32_t>(k) + 1;
  if (kmin == kmax) {  // one distinct value: it is tau and every score ships
    if (threadIdx.x == 0) {
      tau[0] = key_float(kmin);
      if (n_ship) n_ship[0] = static_cast<int32_t>(nv);
    }
    s.pos = 0;
    return s;
  }
  s.pos = 32 - __builtin_clz(kmin ^ kmax);  // bits above pos are shared by every key
  s.mask = s.pos == 32 ? 0u : ~0u << s.pos;
  s.prefix = kmin & s.mask;
  s.need = s.j;
  return s;
}

__device__ __forceinline__ int digit_width(int pos) { return pos < kDigit ? pos : kDigit; }

// One pass's bin choice from the histogram held by the block (thread t:
// bins 2t and 2t + 1); advances the select and, when it is complete, writes
// tau and n_ship. Every thread returns the same state.
__device__ Select select_step(Select s, uint32_t h0, uint32_t h1, CalShared& sh, float* tau, int32_t* n_ship) {
  const int t = threadIdx.x;
  const int w = t / kWave;
  const int lane = t % kWave;
  const int shift = s.pos - digit_width(s.pos);
  const uint32_t c = h0 + h1;
  uint32_t incl = c;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const uint32_t u = __shfl_up(incl, o);
    if (lane >= o) incl += u;
  }
  if (lane == kWave - 1) sh.wcnt[w] = incl;
  __syncthreads();
  uint32_t off = 0;
  for (int v = 0; v < w; ++v) off += sh.wcnt[v];
  incl += off;
  const uint32_t excl = incl - c;
  if (s.need > excl && s.need <= incl) {
    uint32_t r = s.need - excl, b = 2u * t;
    if (r > h0) {
      r -= h0;
      b += 1;
    }
    sh.sel[0] = b;
    sh.sel[1] = r;
  }
  __syncthreads();
  s.prefix |= sh.sel[0] << shift;
  s.need = sh.sel[1];
  s.mask |= ((1u << digit_width(s.pos)) - 1u) << shift;
  s.pos = shift;
  if (s.pos == 0 && t == 0) {
    // The j-th smallest is the need-th of the scores equal to tau: j - need
    // scores lie below it, every other non-NaN score ships.
    tau[0] = key_float(s.prefix);
    if (n_ship) n_ship[0] = static_cast<int32_t>(s.nv - (s.j - s.need));
  }
  // The next writes of wcnt and sel come after two more barriers, which
  // every thread reaches only once it has read them here.
  return s;
}

__device__ __forceinline__ bool in_select(const Select& s, uint32_t key) {
  return (key & s.mask) == s.prefix && key != kNanKey;
}

// Pools of up to kCalRegKeys * kCalBlock scores: one workgroup.
__global__ __launch_bounds__(kCalBlock) void calibrate_kernel(const float* scores, int32_t n, double q, float* tau,
                                                              int32_t* n_ship) {
  __shared__ CalShared sh;
  const int t = threadIdx.x;
  uint32_t keys[kCalRegKeys];
  uint32_t valid = 0, kmin = 0xffffffffu, kmax = 0;
#pragma unroll
  for (int r = 0; r < kCalRegKeys; ++r) {
    const int64_t i = t + static_cast<int64_t>(r) * kCalBlock;
    keys[r] = i < n ? score_key(scores[i]) : kNanKey;
    if (keys[r] != kNanKey) {
      ++valid;
      kmin = min(kmin, keys[r]);
      kmax = max(kmax, keys[r]);
    }
  }
  uint32_t nv;
  block_range(valid, kmin, kmax, sh, nv, kmin, kmax);
  Select s = select_start(nv, kmin, kmax, q, tau, n_ship);
  while (s.pos > 0) {
    const int shift = s.pos - digit_width(s.pos);
    const uint32_t dmask = (1u << digit_width(s.pos)) - 1u;
    sh.hist[t] = 0;
    sh.hist[t + kCalBlock] = 0;
    __syncthreads();
#pragma unroll
    for (int r = 0; r < kCalRegKeys; ++r)
      if (in_select(s, keys[r])) hist_add(sh.hist, (keys[r] >> shift) & dmask);
    __syncthreads();
    s = select_step(s, sh.hist[2 * t], sh.hist[2 * t + 1], sh, tau, n_ship);
  }
}

// ---- larger pools: several workgroups per pass, state in the workspace ----

constexpr int kCalMaxBlocks = 256;

struct CalWs {
  Select sel;
  uint32_t pad[10];
  uint32_t hist[kBins];                // the pass's histogram (zero between passes)
  uint32_t part[kCalMaxBlocks][4];     // per-workgroup count, smallest and largest key
};

// Calls fn(key) for this thread's keys of the pool: kCalRegKeys loads issued
// together per round (one round covers gridDim.x * kCalBlock * kCalRegKeys
// scores, coalesced per load).
template <typename Fn>
__device__ __forceinline__ void for_my_keys(const float* scores, int32_t n, Fn fn) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kCalBlock;
  for (int64_t base = blockIdx.x * static_cast<int64_t>(kCalBlock) + threadIdx.x; base < n;
       base += stride * kCalRegKeys) {
    uint32_t keys[kCalRegKeys];
#pragma unroll
    for (int r = 0; r < kCalRegKeys; ++r) {
      const int64_t i = base + r * stride;
      keys[r] = i < n ? score_key(scores[i]) : kNanKey;
    }
#pragma unroll
    for (int r = 0; r < kCalRegKeys; ++r) fn(keys[r]);
  }
}

__global__ __launch_bounds__(kCalBlock) void calibrate_range_kernel(const float* scores, int32_t n, CalWs* ws) {
  __shared__ CalShared sh;
  uint32_t valid = 0, kmin = 0xffffffffu, kmax = 0;
  for_my_keys(scores, n, [&](uint32_t key) {
    if (key != kNanKey) {
      ++valid;
      kmin = min(kmin, key);
      kmax = max(kmax, key);
    }
  });
  uint32_t nv;
  block_range(valid, kmin, kmax, sh, nv, kmin, kmax);
  if (threadIdx.x == 0) {
    ws->part[blockIdx.x][0] = nv;
    ws->part[blockIdx.x][1] = kmin;
    ws->part[blockIdx.x][2] = kmax;
  }
  if (blockIdx.x == 0) {
    ws->hist[threadIdx.x] = 0;
    ws->hist[threadIdx.x + kCalBlock] = 0;
  }
}

__global__ __launch_bounds__(kCalBlock) void calibrate_init_kernel(CalWs* ws, int blocks, double q, float* tau,
                                                                   int32_t* n_ship) {
  __shared__ CalShared sh;
  const int t = threadIdx.x;
  const bool mine = t < blocks;
  uint32_t nv, kmin, kmax;
  block_range(mine ? ws->part[t][0] : 0u, mine ? ws->part[t][1] : 0xffffffffu, mine ? ws->part[t][2] : 0u, sh, nv,
              kmin, kmax);
  const Select s = select_start(nv, kmin, kmax, q, tau, n_ship);
  if (t == 0) ws->sel = s;
}

__global__ __launch_bounds__(kCalBlock) void calibrate_hist_kernel(const float* scores, int32_t n, CalWs* ws) {
  __shared__ uint32_t h[kBins];
  const Select s = ws->sel;
  if (s.pos == 0) return;
  const int t = threadIdx.x;
  const int shift = s.pos - digit_width(s.pos);
  const uint32_t dmask = (1u << digit_width(s.pos)) - 1u;
  h[t] = 0;
  h[t + kCalBlock] = 0;
  __syncthreads();
  for_my_keys(scores, n, [&](uint32_t key) {
    if (in_select(s, key)) hist_add(h, (key >> shift) & dmask);
  });
  __syncthreads();
  if (h[t]) atomicAdd(&ws->hist[t], h[t]);
  if (h[t + kCalBlock]) atomicAdd(&ws->hist[t + kCalBlock], h[t + kCalBlock]);
}

__global__ __launch_bounds__(kCalBlock) void calibrate_select_kernel(CalWs* ws, float* tau, int32_t* n_ship) {
  __shared__ CalShared sh;
  const int t = threadIdx.x;
  const Select s = ws->sel;
  if (s.pos == 0) return;
  const uint32_t h0 = ws->hist[2 * t], h1 = ws->hist[2 * t + 1];
  ws->hist[2 * t] = 0;  // cleared for the next pass (each thread clears the bins it read)
  ws->hist[2 * t + 1] = 0;
  const Select next = select_step(s, h0, h1, sh, tau, n_ship);
  if (t == 0) ws->sel = next;
}

// At least 4 keys per thread, at most one workgroup per CU.
int calibrate_blocks(int32_t n) {
  const int64_t b = (static_cast<int64_t>(n) + 4 * kCalBlock - 1) / (4 * kCalBlock);
  return static_cast<int>(b < 1 ? 1 : (b > kCalMaxBlocks ? kCalMaxBlocks : b));
}

}  // namespace

size_t calibrate_workspace_bytes(int32_t n) {
  return n > kCalRegKeys * kCalBlock ? sizeof(CalWs) : 0;
}

hipError_t launch_calibrate(const float* scores, int32_t n, double q, float* tau, int32_t* n_ship, void* workspace,
                            hipStream_t stream) {
  if (n <= kCalRegKeys * kCalBlock) {
    calibrate_kernel<<<1, kCalBlock, 0, stream>>>(scores, n, q, tau, n_ship);
    return hipGetLastError();
  }
  CalWs* ws = static_cast<CalWs*>(workspace);
  const int blocks = calibrate_blocks(n);
  calibrate_range_kernel<<<blocks, kCalBlock, 0, stream>>>(scores, n, ws);
  calibrate_init_kernel<<<1, kCalBlock, 0, stream>>>(ws, blocks, q, tau, n_ship);
  for (int pass = 0; pass < 3; ++pass) {  // 32 bits in digits of 11: at most three passes
    calibrate_hist_kernel<<<blocks, kCalBlock, 0, stream>>>(scores, n, ws);
    calibrate_select_kernel<<<1, kCalBlock, 0, stream>>>(ws, tau, n_ship);
  }
  return hipGetLastError();
}

}  // namespace pr
