// C ABI of the verifier library: argument checks, launch-shape selection and
// the streaming state object. Every compute step runs in the kernels of
// row_features.hip, topp.hip and aggregate.hip.
#include <mutex>
#include <new>

#include "aggregate.h"
#include "calibrate.h"
#include "head.h"
#include "topp.h"

using namespace pr;

// Scratch of pr_token_features_noalloc: the split-row partial states of small
// batches, in a file-scope device array instead of a caller's workspace. Each
// GPU the library runs on holds its own copy until the process ends. In host
// code this name is only a stand-in for the symbol: its device address comes
// from hipGetSymbolAddress (see noalloc_scratch below), never from the name.
static __device__ __align__(256) unsigned char scratch[PR_NOALLOC_SCRATCH_BYTES];

struct pr_stream {
  int device;
  StreamDev dev;
  pr_agg_params params;
  Partial* ws;  // split-row workspace for up to max_slots rows of kStreamMaxSplit workgroups
  void* block;  // single allocation backing everything above
};

namespace {

constexpr int kStreamMaxSplit = 32;
// The top-p histogram packs a bin's count into 24 bits.
constexpr int32_t kTopPMaxVocab = 1 << 24;

inline hipStream_t as_stream(void* s) { return static_cast<hipStream_t>(s); }

inline bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

inline size_t dtype_size(pr_dtype d) { return d == PR_BF16 ? 2 : 4; }

bool features_complete(const pr_token_features_t* o) {
  return o && o->max_logit && o->lse && o->entropy && o->logprob && o->maxprob && o->margin && o->rank &&
         o->argmax && o->cutoff && o->flags;
}

pr_status check_rows(const void* logits, pr_dtype dtype, int64_t n_rows, int32_t V, int64_t row_stride,
                     const int32_t* ids, const float* temps) {
  if (dtype != PR_F32 && dtype != PR_BF16) return PR_ERR_INVALID_ARG;
  if (n_rows < 0 || V < 2 || row_stride < V) return PR_ERR_INVALID_ARG;
  if (n_rows > 0 && (!logits || !ids || !temps)) return PR_ERR_INVALID_ARG;
  if (logits && !aligned(logits, dtype_size(dtype))) return PR_ERR_INVALID_ARG;
  // Grid limits: rows * split must stay far below 2^31 workgroups.
  if (n_rows > (int64_t{1} << 26)) return PR_ERR_UNSUPPORTED;
  return PR_OK;
}

pr_status hip_status(hipError_t e) {
  if (e == hipSuccess) return PR_OK;
  if (e == hipErrorOutOfMemory) return PR_ERR_NO_MEMORY;
  if (e == hipErrorNotSupported) return PR_ERR_UNSUPPORTED;
  return PR_ERR_HIP;
}

pr_agg_params default_params() {
  pr_agg_params p;
  p.q = 0.1;
  for (double& w : p.w) w = 0.0;
  p.w[1] = 1.0;  // mean(maxprob)
  p.b = 0.0;
  p.link = 0;
  return p;
}

// Device address of `scratch` on the device that runs `stream` (the current
// device for the NULL stream), looked up once per device with that device
// current and kept. No allocation happens here or later.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

pr_status noalloc_scratch(hipStream_t stream, void** out) {
  int cur = 0;
  if (hipGetDevice(&cur) != hipSuccess) return PR_ERR_HIP;
  int dev = cur;
  if (stream) {
    hipDevice_t d = 0;
    if (hipStreamGetDevice(stream, &d) != hipSuccess) return PR_ERR_HIP;
    dev = static_cast<int>(d);
  }
  if (dev < 0 || dev >= kMaxDevices) return PR_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    if (dev != cur && hipSetDevice(dev) != hipSuccess) return PR_ERR_HIP;
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (dev != cur && hipSetDevice(cur) != hipSuccess) return PR_ERR_HIP;
    if (e != hipSuccess || !p) return PR_ERR_HIP;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return PR_OK;
}

bool params_ok(const pr_agg_params& p) {
  if (!(p.q >= 0.0 && p.q <= 1.0)) return false;
  if (p.link != 0 && p.link != 1) return false;
  return true;
}

}  // namespace

extern "C" {

const char* pr_status_string(pr_status status) {
  switch (status) {
    case PR_OK:
      return "ok";
    case PR_ERR_INVALID_ARG:
      return "invalid argument";
    case PR_ERR_UNSUPPORTED:
      return "unsupported";
    case PR_ERR_HIP:
      return "HIP runtime error";
    case PR_ERR_NO_MEMORY:
      return "out of device memory";
  }
  return "unknown status";
}

void pr_agg_params_default(pr_agg_params* params) {
  if (params) *params = default_params();
}

size_t pr_token_features_workspace(pr_dtype dtype, int64_t n_rows, int32_t vocab, int32_t top_p_on) {
  if (n_rows <= 0 || vocab < 2) return 0;
  if (top_p_on) return topp_workspace(dtype, n_rows, vocab);
  return split_workspace_bytes(n_rows, row_split(n_rows, vocab, dtype));
}

pr_status pr_token_features(const void* logits, pr_dtype dtype, int64_t n_rows, int32_t vocab,
                            int64_t row_stride, const int32_t* sampled_ids, const float* temperature,
                            const float* top_p, const pr_token_features_t* out, void* workspace,
                            size_t workspace_bytes, void* stream) {
  pr_status st = check_rows(logits, dtype, n_rows, vocab, row_stride, sampled_ids, temperature);
  if (st != PR_OK) return st;
  if (!features_complete(out)) return PR_ERR_INVALID_ARG;
  const size_t need = pr_token_features_workspace(dtype, n_rows, vocab, top_p ? 1 : 0);
  if (need > 0 && (!workspace || workspace_bytes < need || !aligned(workspace, 16))) return PR_ERR_INVALID_ARG;
  if (n_rows == 0) return PR_OK;
  RowArgs a{};
  a.logits = logits;
  a.n_rows = n_rows;
  a.V = vocab;
  a.row_stride = row_stride;
  a.sampled_ids = sampled_ids;
  a.temperature = temperature;
  a.top_p = top_p;
  a.out = *out;
  if (top_p && vocab >= kTopPMaxVocab) return PR_ERR_UNSUPPORTED;
  if (top_p) return hip_status(launch_topp(a, dtype, workspace, as_stream(stream)));
  a.G = row_split(n_rows, vocab, dtype);
  a.ws = static_cast<Partial*>(workspace);
  return hip_status(launch_row_features(a, dtype, as_stream(stream)));
}

pr_status pr_token_features_noalloc(const void* logits, pr_dtype dtype, int64_t n_rows, int32_t vocab,
                                    int64_t row_stride, const int32_t* sampled_ids, const float* temperature,
                                    const float* top_p, const pr_token_features_t* out, void* stream) {
  pr_status st = check_rows(logits, dtype, n_rows, vocab, row_stride, sampled_ids, temperature);
  if (st != PR_OK) return st;
  if (!features_complete(out)) return PR_ERR_INVALID_ARG;
  const size_t need = pr_token_features_workspace(dtype, n_rows, vocab, top_p ? 1 : 0);
  if (need > PR_NOALLOC_SCRATCH_BYTES) return PR_ERR_UNSUPPORTED;
  if (n_rows == 0) return PR_OK;
  void* ws = nullptr;
  if (need > 0) {
    st = noalloc_scratch(as_stream(stream), &ws);
    if (st != PR_OK) return st;
  }
  return pr_token_features(logits, dtype, n_rows, vocab, row_stride, sampled_ids, temperature, top_p, out, ws,
                           need, stream);
}

pr_status pr_feature_sequence(const void* logits, pr_dtype dtype, int64_t n_rows, int32_t vocab,
                              int64_t row_stride, const int32_t* sampled_ids, const float* temperature,
                              const float* top_p, const int32_t* offsets, int32_t n_req, int32_t top_k,
                              float* X, const pr_token_features_t* features, void* stream) {
  pr_status st = check_rows(logits, dtype, n_rows, vocab, row_stride, sampled_ids, temperature);
  if (st != PR_OK) return st;
  if (top_k < 1 || top_k > PR_MAX_TOP_K || n_req < 0) return PR_ERR_INVALID_ARG;
  if (features && !features_complete(features)) return PR_ERR_INVALID_ARG;
  if (n_rows == 0) return PR_OK;
  if (n_req == 0 || !offsets || !X || !aligned(X, 16)) return PR_ERR_INVALID_ARG;
  RowArgs a{};
  a.logits = logits;
  a.n_rows = n_rows;
  a.V = vocab;
  a.row_stride = row_stride;
  a.sampled_ids = sampled_ids;
  a.temperature = temperature;
  a.top_p = top_p;
  if (features) a.out = *features;
  a.G = 1;
  a.X = X;
  a.offsets = offsets;
  a.n_req = n_req;
  a.top_k = top_k;
  if (top_p && vocab >= kTopPMaxVocab) return PR_ERR_UNSUPPORTED;
  if (top_p) return hip_status(launch_topp(a, dtype, nullptr, as_stream(stream)));
  return hip_status(launch_feature_sequence(a, dtype, as_stream(stream)));
}

pr_status pr_sample_features(const void* logits, pr_dtype dtype, int64_t n_rows, int32_t vocab, int64_t row_stride,
                             const float* temperature, uint64_t seed, uint64_t offset, int32_t* sampled_ids,
                             const pr_token_features_t* features, const int32_t* offsets, int32_t n_req,
                             int32_t top_k, float* X, void* stream) {
  if (dtype != PR_F32 && dtype != PR_BF16) return PR_ERR_INVALID_ARG;
  if (n_rows < 0 || vocab < 2 || row_stride < vocab) return PR_ERR_INVALID_ARG;
  if (n_rows > (int64_t{1} << 26)) return PR_ERR_UNSUPPORTED;
  if (features && !features_complete(features)) return PR_ERR_INVALID_ARG;
  if (X && (top_k < 1 || top_k > PR_MAX_TOP_K || n_req < 0)) return PR_ERR_INVALID_ARG;
  if (n_rows == 0) return PR_OK;
  if (!logits || !temperature || !sampled_ids || !aligned(logits, dtype_size(dtype))) return PR_ERR_INVALID_ARG;
  if (X && (n_req == 0 || !offsets || !aligned(X, 16))) return PR_ERR_INVALID_ARG;
  RowArgs a{};
  a.logits = logits;
  a.n_rows = n_rows;
  a.V = vocab;
  a.row_stride = row_stride;
  a.sampled_ids = nullptr;
  a.temperature = temperature;
  if (features) a.out = *features;
  a.G = 1;
  a.X = X;
  a.offsets = offsets;
  a.n_req = n_req;
  a.top_k = top_k;
  a.sampled_out = sampled_ids;
  // One key per (seed, offset): the offset is spread by an odd multiplier
  // (a bijection of 64-bit words), so each offset gives its own key.
  const uint64_t key = seed ^ (offset * 0x9E3779B97F4A7C15ull);
  a.key0 = static_cast<uint32_t>(key);
  a.key1 = static_cast<uint32_t>(key >> 32);
  return hip_status(launch_sample(a, dtype, as_stream(stream)));
}

size_t pr_verifier_head_workspace(int64_t n_rows) { return n_rows > 0 ? head_workspace_bytes(n_rows) : 0; }

pr_status pr_verifier_head(const float* X, int64_t n_rows, const int32_t* offsets, int32_t n_req, int32_t max_len,
                           const float* weights, float* scores, void* workspace, size_t workspace_bytes,
                           void* stream) {
  if (n_rows < 0 || n_req < 0 || max_len < 1) return PR_ERR_INVALID_ARG;
  if (n_rows > (int64_t{1} << 30) || max_len > (1 << 20)) return PR_ERR_UNSUPPORTED;  // grid limits
  if (n_req == 0) return PR_OK;
  if (!offsets || !weights || !scores || !aligned(weights, 16)) return PR_ERR_INVALID_ARG;
  if (n_rows > 0 && (!X || !aligned(X, 4))) return PR_ERR_INVALID_ARG;
  const size_t need = pr_verifier_head_workspace(n_rows);
  if (need > 0 && (!workspace || workspace_bytes < need || !aligned(workspace, 16))) return PR_ERR_INVALID_ARG;
  HeadArgs a{};
  a.X = X;
  a.n_rows = n_rows;
  a.offsets = offsets;
  a.n_req = n_req;
  a.max_len = max_len;
  a.weights = weights;
  a.scores = scores;
  a.ws = static_cast<float*>(workspace);
  return hip_status(launch_head(a, as_stream(stream)));
}

pr_status pr_request_aggregate(const pr_token_features_t* feats, const int32_t* offsets, int32_t n_req,
                               const pr_agg_params* params, const pr_request_agg_t* out, void* stream) {
  if (n_req < 0 || !out) return PR_ERR_INVALID_ARG;
  if (n_req == 0) return PR_OK;
  if (!feats || !offsets || !feats->logprob || !feats->maxprob || !feats->entropy || !feats->margin)
    return PR_ERR_INVALID_ARG;
  const pr_agg_params p = params ? *params : default_params();
  if (!params_ok(p)) return PR_ERR_INVALID_ARG;
  return hip_status(launch_aggregate(*feats, offsets, n_req, p, *out, as_stream(stream)));
}

pr_status pr_route(const float* scores, int32_t n_req, float threshold, uint8_t* ship, int32_t* n_ship,
                   void* stream) {
  if (n_req < 0) return PR_ERR_INVALID_ARG;
  if (n_req > 0 && (!scores || !ship)) return PR_ERR_INVALID_ARG;
  if (n_req == 0 && !n_ship) return PR_OK;
  return hip_status(launch_route(scores, n_req, threshold, ship, n_ship, as_stream(stream)));
}

size_t pr_calibrate_workspace(int32_t n) { return n < 0 ? 0 : calibrate_workspace_bytes(n); }

pr_status pr_calibrate_threshold(const float* scores, int32_t n, double ship_fraction, float* tau, int32_t* n_ship,
                                 void* workspace, size_t workspace_bytes, void* stream) {
  if (n < 0 || !tau || (n > 0 && !scores)) return PR_ERR_INVALID_ARG;
  if (!(ship_fraction >= 0.0 && ship_fraction <= 1.0)) return PR_ERR_INVALID_ARG;
  const size_t need = calibrate_workspace_bytes(n);
  if (need && (!workspace || workspace_bytes < need || reinterpret_cast<uintptr_t>(workspace) % 4 != 0))
    return PR_ERR_INVALID_ARG;
  return hip_status(launch_calibrate(scores, n, ship_fraction, tau, n_ship, workspace, as_stream(stream)));
}

pr_status pr_validate_offsets(const int32_t* offsets, int32_t n_req, int64_t n_rows, void* stream) {
  if (!offsets || n_req < 0) return PR_ERR_INVALID_ARG;
  int32_t* host = new (std::nothrow) int32_t[static_cast<size_t>(n_req) + 1];
  if (!host) return PR_ERR_NO_MEMORY;
  hipError_t e = hipMemcpyAsync(host, offsets, (static_cast<size_t>(n_req) + 1) * sizeof(int32_t),
                                hipMemcpyDeviceToHost, as_stream(stream));
  if (e == hipSuccess) e = hipStreamSynchronize(as_stream(stream));
  pr_status st = hip_status(e);
  if (st == PR_OK) {
    if (host[0] != 0 || host[n_req] != n_rows) st = PR_ERR_INVALID_ARG;
    for (int32_t i = 0; st == PR_OK && i < n_req; ++i)
      if (host[i + 1] < host[i]) st = PR_ERR_INVALID_ARG;
  }
  delete[] host;
  return st;
}

pr_status pr_stream_create(int32_t max_slots, int32_t max_len, const pr_agg_params* params, pr_stream** state) {
  if (!state || max_slots <= 0 || max_len < 0) return PR_ERR_INVALID_ARG;
  *state = nullptr;
  const pr_agg_params p = params ? *params : default_params();
  if (!params_ok(p)) return PR_ERR_INVALID_ARG;
  const size_t S = static_cast<size_t>(max_slots);
  const size_t L = static_cast<size_t>(max_len);
  auto up = [](size_t b) { return (b + 255) & ~size_t{255}; };
  const size_t b_ws = up(split_workspace_bytes(static_cast<int64_t>(S), kStreamMaxSplit));
  const size_t b_sum = up(S * 4 * sizeof(double));
  const size_t b_hist = up(S * 4 * L * sizeof(float));
  const size_t b_min = up(S * 4 * sizeof(float));
  const size_t b_cnt = up(S * sizeof(int32_t));
  const size_t b_nan = up(S * sizeof(uint32_t));
  const bool bounded = max_len == 0;  // P-square markers instead of the history
  const size_t b_p2q = bounded ? up(S * 20 * sizeof(double)) : 0;
  const size_t b_p2n = bounded ? up(S * 16 * sizeof(int32_t)) : 0;
  const size_t total = b_ws + b_sum + b_hist + b_min + b_cnt + b_nan + b_p2q + b_p2n;
  pr_stream* s = new (std::nothrow) pr_stream();
  if (!s) return PR_ERR_NO_MEMORY;
  hipError_t e = hipGetDevice(&s->device);
  if (e == hipSuccess) e = hipMalloc(&s->block, total);
  if (e != hipSuccess) {
    delete s;
    return hip_status(e);
  }
  char* b = static_cast<char*>(s->block);
  s->ws = reinterpret_cast<Partial*>(b);
  b += b_ws;
  s->dev.sum = reinterpret_cast<double*>(b);
  b += b_sum;
  s->dev.hist = reinterpret_cast<float*>(b);
  b += b_hist;
  s->dev.minv = reinterpret_cast<float*>(b);
  b += b_min;
  s->dev.count = reinterpret_cast<int32_t*>(b);
  b += b_cnt;
  s->dev.nanbits = reinterpret_cast<uint32_t*>(b);
  b += b_nan;
  s->dev.p2q = bounded ? reinterpret_cast<double*>(b) : nullptr;
  b += b_p2q;
  s->dev.p2n = bounded ? reinterpret_cast<int32_t*>(b) : nullptr;
  s->dev.p2p = p.q;
  if (bounded) s->dev.hist = nullptr;
  s->dev.max_slots = max_slots;
  s->dev.max_len = max_len;
  s->params = p;
  e = launch_stream_clear(s->dev, nullptr, 0, nullptr);
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e != hipSuccess) {
    (void)hipFree(s->block);
    delete s;
    return hip_status(e);
  }
  *state = s;
  return PR_OK;
}

pr_status pr_stream_step(pr_stream* state, const void* logits, pr_dtype dtype, int32_t n_active, int32_t vocab,
                         int64_t row_stride, const int32_t* slot_ids, const int32_t* sampled_ids,
                         const float* temperature, const float* top_p, const pr_token_features_t* out,
                         void* stream) {
  if (!state) return PR_ERR_INVALID_ARG;
  pr_status st = check_rows(logits, dtype, n_active, vocab, row_stride, sampled_ids, temperature);
  if (st != PR_OK) return st;
  if (n_active > state->dev.max_slots) return PR_ERR_INVALID_ARG;
  if (n_active > 0 && !slot_ids) return PR_ERR_INVALID_ARG;
  if (top_p && vocab >= kTopPMaxVocab) return PR_ERR_UNSUPPORTED;
  if (out && !features_complete(out)) return PR_ERR_INVALID_ARG;
  if (n_active == 0) return PR_OK;
  RowArgs a{};
  a.logits = logits;
  a.n_rows = n_active;
  a.V = vocab;
  a.row_stride = row_stride;
  a.sampled_ids = sampled_ids;
  a.temperature = temperature;
  a.top_p = top_p;
  if (out) a.out = *out;
  int G = row_split(n_active, vocab, dtype);
  if (G > kStreamMaxSplit) G = kStreamMaxSplit;
  a.G = G;
  a.ws = state->ws;
  a.slot_ids = slot_ids;
  a.st = state->dev;
  if (top_p) return hip_status(launch_topp(a, dtype, nullptr, as_stream(stream)));
  return hip_status(launch_row_features(a, dtype, as_stream(stream)));
}

pr_status pr_stream_finish(pr_stream* state, const int32_t* slots, int32_t n, float threshold,
                           const pr_request_agg_t* out, uint8_t* ship, void* stream) {
  if (!state || n < 0) return PR_ERR_INVALID_ARG;
  if (n == 0) return PR_OK;
  if (!slots) return PR_ERR_INVALID_ARG;
  pr_request_agg_t o{};
  if (out) o = *out;
  return hip_status(
      launch_stream_finish(state->dev, slots, n, state->params, threshold, o, ship, as_stream(stream)));
}

pr_status pr_stream_reset_slots(pr_stream* state, const int32_t* slots, int32_t n, void* stream) {
  if (!state || n < 0) return PR_ERR_INVALID_ARG;
  if (n == 0) return PR_OK;
  if (!slots) return PR_ERR_INVALID_ARG;
  return hip_status(launch_stream_clear(state->dev, slots, n, as_stream(stream)));
}

void pr_stream_destroy(pr_stream* state) {
  if (!state) return;
  int prev = 0;
  (void)hipGetDevice(&prev);
  (void)hipSetDevice(state->device);
  (void)hipDeviceSynchronize();
  (void)hipFree(state->block);
  (void)hipSetDevice(prev);
  delete state;
}

}  // extern "C"
