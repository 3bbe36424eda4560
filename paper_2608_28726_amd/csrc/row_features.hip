// Vocabulary-row reduction: per-token confidence features in one pass over
// each logit row (Pro-Router, Sec. 3.1, Eq. 3, extended to max logit,
// logsumexp, entropy, log-probability, top-1/top-2 margin and rank of the
// sampled token, after temperature).
//
// One or more workgroups stream a row with 16-byte loads. Every lane keeps
// an online (max, sum 2^x, sum 2^x * x) state in base 2 with exponent
// argument x = z * log2(e)/T - a (a = the lane's running max times
// log2(e)/T), the top-1 value/index and top-2 value, and the number of
// tokens that precede the sampled token y in the order "larger logit first,
// equal logits by lower index". Comparisons use the raw logits, so
// temperature scaling cannot create false ties. Lanes merge with wave
// shuffles, waves through LDS; a row split over G workgroups merges the G
// partial states either in a second kernel or in the last workgroup to
// finish (streaming decode).
#include "row_scan.h"

namespace pr {

using namespace scan;

// MODE 0: one workgroup per row, finalised in place.
// MODE 1: G workgroups per row write partial states to a.ws.
// MODE 2: streaming; G workgroups per row, the last to finish merges,
//         finalises and updates the request slot.
// Occupancy target: 8 waves per SIMD keep enough loads in flight.
#ifndef PR_ROW_WAVES_PER_EU
#define PR_ROW_WAVES_PER_EU 8
#endif

template <typename Tin, int BLOCK, int U, int MODE>
__global__ __launch_bounds__(BLOCK) __attribute__((amdgpu_waves_per_eu(PR_ROW_WAVES_PER_EU)))
void row_features_kernel(RowArgs a) {
  const int G = a.G;
  const int64_t r = blockIdx.x / G;
  const int g = blockIdx.x % G;
  if (r >= a.n_rows) return;
  constexpr int VEC = Elem<Tin>::kVec;
  const void* row = static_cast<const Tin*>(a.logits) + r * a.row_stride;
  const RowCtx cx = row_ctx<Tin>(a, r, row);
  const int64_t nvec = (a.V - cx.h) / VEC;
  const int64_t vb = nvec * g / G;
  const int64_t ve = nvec * (g + 1) / G;

  Lane L;
  lane_init(L);
  scan_stretch<Tin, BLOCK, U>(row, a.V, vb, ve, g == 0, g == G - 1, nvec, cx, L);
  Partial p = block_merge<BLOCK>(L, cx.c);

  __shared__ int sh_last;
  __shared__ Partial sh_p;
  if (MODE == 1) {
    if (threadIdx.x == 0) a.ws[r * G + g] = p;
    return;
  }
  if (MODE == 2 && G > 1) {
    if (threadIdx.x == 0) {
      a.ws[r * G + g] = p;
      __threadfence();
      const uint32_t old = atomicAdd(&a.counters[r], 1u);
      sh_last = (old == static_cast<uint32_t>(G - 1));
    }
    __syncthreads();
    if (!sh_last) return;
    __threadfence();
    if (threadIdx.x == 0) {
      sh_p = merge_partials(a.ws + r * G, G, cx.c);
      a.counters[r] = 0u;
    }
    __syncthreads();
    p = sh_p;
  }
  const uint32_t fix = rank_fixup<Tin, BLOCK>(row, a.V, nvec, cx);
  if (threadIdx.x == 0) {
    float conf[4];
    finalize_row(a, r, p, cx, fix, conf);
    if (MODE == 2) stream_update(a.st, a.slot_ids[r], conf);
  }
}

// Second kernel of MODE 1: merges each row's G partials and finalises.
template <typename Tin, int BLOCK>
__global__ __launch_bounds__(BLOCK) void row_merge_kernel(RowArgs a) {
  const int64_t r = blockIdx.x;
  if (r >= a.n_rows) return;
  constexpr int VEC = Elem<Tin>::kVec;
  const void* row = static_cast<const Tin*>(a.logits) + r * a.row_stride;
  const RowCtx cx = row_ctx<Tin>(a, r, row);
  const int64_t nvec = (a.V - cx.h) / VEC;
  const uint32_t fix = rank_fixup<Tin, BLOCK>(row, a.V, nvec, cx);
  if (threadIdx.x == 0) {
    const Partial p = merge_partials(a.ws + r * a.G, a.G, cx.c);
    float conf[4];
    finalize_row(a, r, p, cx, fix, conf);
  }
}

namespace {

#ifndef PR_ROW_BLOCK
#define PR_ROW_BLOCK 128
#endif
#ifndef PR_UNROLL_BF16
#define PR_UNROLL_BF16 2
#endif
#ifndef PR_UNROLL_F32
#define PR_UNROLL_F32 4
#endif

constexpr int kBlock = PR_ROW_BLOCK;
constexpr int kTargetBlocks = 2048;  // 8 workgroups per CU on 256 CUs
constexpr int kMaxSplit = 64;

// 16-byte vectors per lane per loop step.
template <typename Tin>
constexpr int unroll_for() {
  return Elem<Tin>::kVec == 8 ? PR_UNROLL_BF16 : PR_UNROLL_F32;
}

}  // namespace

int row_split(int64_t n_rows, int32_t V, pr_dtype dtype) {
  const int VEC = dtype == PR_BF16 ? 8 : 4;
  const int64_t nvec = V / VEC;
  if (n_rows <= 0 || n_rows >= kTargetBlocks) return 1;
  int64_t G = (kTargetBlocks + n_rows - 1) / n_rows;
  const int64_t by_work = nvec / (kBlock * 4);  // at least ~4 vectors per lane
  if (G > by_work) G = by_work;
  if (G > kMaxSplit) G = kMaxSplit;
  if (G < 1) G = 1;
  return static_cast<int>(G);
}

template <typename Tin>
static hipError_t launch_typed(const RowArgs& a, int mode, hipStream_t stream) {
  constexpr int U = unroll_for<Tin>();
  const dim3 grid(static_cast<unsigned>(a.n_rows * a.G));
  if (mode == 2) {
    row_features_kernel<Tin, kBlock, U, 2><<<grid, kBlock, 0, stream>>>(a);
  } else if (a.G == 1) {
    row_features_kernel<Tin, kBlock, U, 0><<<grid, kBlock, 0, stream>>>(a);
  } else {
    row_features_kernel<Tin, kBlock, U, 1><<<grid, kBlock, 0, stream>>>(a);
    row_merge_kernel<Tin, kWave><<<dim3(static_cast<unsigned>(a.n_rows)), kWave, 0, stream>>>(a);
  }
  return hipGetLastError();
}

hipError_t launch_row_features(const RowArgs& a, pr_dtype dtype, int mode, hipStream_t stream) {
  if (a.n_rows == 0) return hipSuccess;
  return dtype == PR_BF16 ? launch_typed<uint16_t>(a, mode, stream) : launch_typed<float>(a, mode, stream);
}

}  // namespace pr
