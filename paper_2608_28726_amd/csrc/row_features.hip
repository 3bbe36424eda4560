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
// partial states in a second kernel, which also updates the streaming
// decode state.
#include <type_traits>

#include "p2.h"
#include "row_scan.h"
#include "sample.h"
#include "topk.h"

namespace pr {

using namespace scan;

// Occupancy target of the one-row-per-workgroup kernel: 5 waves per SIMD
// leave the registers of two load buffers and the rarely taken top-2
// tournament without spilling.
#ifndef PR_ROW_WAVES_PER_EU
#define PR_ROW_WAVES_PER_EU 5
#endif

// SPLIT == false: one workgroup per row, finalised in place (and, when
// slot ids are given, the row's token joins its request slot).
// SPLIT == true: G workgroups per row write partial states to a.ws; the
// merge kernel below finalises. Kernel boundaries make the partials visible,
// so no workgroup waits or fences on another.
// SEQ == true (one workgroup per row): the row's K largest logits are found
// in the same pass and row r of the verifier input sequence X is written.
// SAMPLE == true (one workgroup per row): the row's token is drawn in the
// same pass (sample.h) and the row is finalised for it.
template <typename Tin, int BLOCK, int U, int LD, bool SPLIT, bool SEQ = false, bool SAMPLE = false>
__global__ __launch_bounds__(BLOCK)
__attribute__((amdgpu_waves_per_eu(BLOCK >= 512 ? BLOCK / 256 : PR_ROW_WAVES_PER_EU)))
void row_features_kernel(RowArgs a) {
  static_assert(!(SPLIT && SEQ), "the sequence variant keeps a row in one workgroup");
  static_assert(!(SPLIT && SAMPLE), "the sampling variant keeps a row in one workgroup");
  const int G = a.G;
  const int64_t r = blockIdx.x / G;
  const int g = blockIdx.x % G;
  if (r >= a.n_rows) return;
  constexpr int VEC = Elem<Tin>::kVec;
  const void* row = static_cast<const Tin*>(a.logits) + r * a.row_stride;
  const int64_t h = head_elems<Tin>(row, a.V);
  const int64_t nvec = (a.V - h) / VEC;
  const int64_t vb = nvec * g / G;
  const int64_t ve = nvec * (g + 1) / G;
  vec4u v[LD];
  stretch_prefetch<Tin, BLOCK, LD>(row, h, vb, ve, v);
  const RowCtx cx = row_ctx<Tin>(a, r, row);
  // Wide workgroups (one row per CU) read the slot state early so that its
  // latency hides behind the row; narrow ones read it at the end, where
  // other workgroups on the CU cover it and no registers stay tied up.
  constexpr bool kEarlySlot = !SPLIT && BLOCK >= 512;
  SlotState ss{-1};
  p2::RowMarkers pm;
  if (kEarlySlot) {
    ss = slot_load(a, r);
    if (threadIdx.x < kWave) pm.fetch(a, r);
  }

  Lane L;
  lane_init(L);
  using SeqHook = typename std::conditional<SEQ, topk::Hook, NoHook>::type;
  typename std::conditional<SAMPLE, HookPair<sample::Hook, SeqHook>, SeqHook>::type hook;
  SeqHook& seq_hook = [&]() -> SeqHook& {
    if constexpr (SAMPLE) return hook.b;
    else return hook;
  }();
  if constexpr (SEQ) seq_hook.init();
  if constexpr (SAMPLE) hook.a.init(a.key0, a.key1, r);
  // Workgroups of 512 or more threads run one per CU: there the bucket of
  // each lane's maximum is kept in registers rather than read back at the end.
  scan_stretch<Tin, BLOCK, U, LD, (BLOCK >= 512)>(row, a.V, vb, ve, g == 0, g == G - 1, nvec, cx, L, v, hook);
  const Partial p = block_merge<BLOCK>(L, cx.c);
  if (SPLIT) {
    if (threadIdx.x == 0) a.ws[r * G + g] = p;
    if (g == 0) {  // the row's context and rank corrections for the merge
      const uint32_t fix = rank_fixup<Tin, BLOCK>(row, a.V, nvec, cx);
      if (threadIdx.x == 0) split_meta(a.ws, a.n_rows, G)[r] = RowMeta{cx.T, cx.zy, cx.y, fix};
    }
    return;
  }
  const uint32_t fix = rank_fixup<Tin, BLOCK>(row, a.V, nvec, cx);
  RowCtx cf = cx;  // the context the row is finalised with
  if constexpr (SAMPLE) {
    // The token drawn for the row; its rank is not counted (that needs its
    // value before the pass), and is written as -1, "not available".
    __shared__ sample::Shared ssh;
    __shared__ float sh_ref;
    __shared__ uint32_t sh_def;
    if (threadIdx.x == 0) {  // the merged state p is valid in the first wave
      sh_ref = p.m * cx.c;
      sh_def = (row_flags(a, r, p, cx.T) & (PR_FLAG_NONFINITE | PR_FLAG_BAD_TP)) == 0 ? 1u : 0u;
    }
    __syncthreads();
    sample::pick<Tin, BLOCK, U>(row, nvec, cx, L, hook.a, sh_ref, sh_def != 0, ssh, cf.y, cf.zy);
  }
  if constexpr (SEQ) {
    __shared__ topk::Store<BLOCK> ts;
    const topk::Lds lds = ts.view();
    // inline: out of line its LDS is reached through flat addresses
    [[clang::always_inline]] topk::select_topk<Tin, BLOCK, U>(row, a.V, cx.h, vb, ve, nvec, a.top_k, seq_hook, lds);
    if (threadIdx.x < kWave) {  // the merged state p is valid in the first wave
      const float H = topk::topk_entropy_f32(lds.top, a.top_k, p.m, cx.c, p.S);
      const float rho = topk::position_fraction(a.offsets, a.n_req, r);
      if (threadIdx.x == 0) {
        float conf[4];
        const uint32_t flags = finalize_row(a, r, p, cf, fix, conf);
        write_sequence_row(a, r, conf, flags, H, rho);
        if (SAMPLE) {
          a.sampled_out[r] = cf.y;
          if (a.out.rank) a.out.rank[r] = -1;
        }
      }
    }
    return;
  }
  if (threadIdx.x < kWave) {
    if (!kEarlySlot) pm.fetch(a, r);
    float conf[4];
    if (threadIdx.x == 0) {
      finalize_row(a, r, p, cf, fix, conf);
      stream_update(a.st, kEarlySlot ? ss : slot_load(a, r), conf);
      if (SAMPLE) {
        a.sampled_out[r] = cf.y;
        if (a.out.rank) a.out.rank[r] = -1;
      }
    }
    if (pm.slot >= 0) p2::feed_row(a, pm, conf);
  }
}

// Merges each row's G partial states and finalises the row: one wave per
// row, lane g holding partial g (G <= 64). Every input (the partials, the
// row's context record and the slot state) is loaded at once, so the merge
// costs one memory round trip.
__global__ __launch_bounds__(kWave) void row_merge_kernel(RowArgs a) {
  const int64_t r = blockIdx.x;
  if (r >= a.n_rows) return;
  const int G = a.G;
  const int lane = threadIdx.x;
  Partial q;
  if (lane < G) {
    q = a.ws[r * G + lane];
  } else {
    q.m = -INFINITY;
    q.S = 0.0f;
    q.E = 0.0f;
    q.t1 = -INFINITY;
    q.t1i = kNoIndex;
    q.t2 = -INFINITY;
    q.cnt = 0;
    q.pad = 0;
  }
  const RowMeta meta = split_meta(a.ws, a.n_rows, G)[r];
  const SlotState ss = slot_load(a, r);
  p2::RowMarkers pm;
  pm.fetch(a, r);
  RowCtx cx;
  cx.T = meta.T;
  cx.c = temperature_ok(meta.T) ? kLog2e / meta.T : kLog2e;
  cx.zy = meta.zy;
  cx.y = meta.y;
  cx.fix_vec = 0;
  cx.h = 0;
  cx.thr_before = 0.0f;
  cx.thr_lo = 0.0f;
  Partial p;
  p.m = wave_max(q.m);
  rebase(q.m == -INFINITY, q.m * cx.c, p.m * cx.c, q.S, q.E);
  p.S = wave_sum(q.S);
  p.E = wave_sum(q.E);
  wave_top2(q.t1, q.t1i, q.t2);
  p.t1 = q.t1;
  p.t1i = q.t1i;
  p.t2 = q.t2;
  p.cnt = wave_sum_u(q.cnt);
  p.pad = 0;
  float conf[4];
  if (lane == 0) {
    finalize_row(a, r, p, cx, meta.fix, conf);
    stream_update(a.st, ss, conf);
  }
  if (pm.slot >= 0) p2::feed_row(a, pm, conf);
}

namespace {

#ifndef PR_UNROLL_BF16
#define PR_UNROLL_BF16 2
#endif
#ifndef PR_UNROLL_F32
#define PR_UNROLL_F32 4
#endif
// Load depth LD of the one-row-per-workgroup kernel: with double buffering
// each lane keeps between LD and 2 * LD 16-byte loads in flight.
#ifndef PR_LOAD_DEPTH_BF16
#define PR_LOAD_DEPTH_BF16 2
#endif
#ifndef PR_LOAD_DEPTH_F32
#define PR_LOAD_DEPTH_F32 4
#endif

// Workgroup of the one-row-per-workgroup tier (batches of kWideRows rows or
// more) in every variant: four waves per row read the 64-request batch at
// 6.6 TB/s against 6.4 for two in the plain features pass, and the sequence
// and sampling variants gain 1-2 % as well.
#ifndef PR_FEAT_BLOCK
#define PR_FEAT_BLOCK 256
#endif
constexpr int kFeatBlock = PR_FEAT_BLOCK;
constexpr int kMaxSplit = 64;

// 16-byte vectors per lane per loop step.
template <typename Tin>
constexpr int unroll_for() {
  return Elem<Tin>::kVec == 8 ? PR_UNROLL_BF16 : PR_UNROLL_F32;
}
template <typename Tin>
constexpr int load_depth_for() {
  return Elem<Tin>::kVec == 8 ? PR_LOAD_DEPTH_BF16 : PR_LOAD_DEPTH_F32;
}

}  // namespace

#ifndef PR_WIDE_ROWS
#define PR_WIDE_ROWS 2048
#endif
#ifndef PR_WIDE_BLOCK
#define PR_WIDE_BLOCK 1024
#endif
#ifndef PR_MID_BLOCK
#define PR_MID_BLOCK 256
#endif
#ifndef PR_SPLIT_BLOCK
#define PR_SPLIT_BLOCK 512
#endif
// Workgroup size by batch size: below kWideRows rows a row gets one wider
// workgroup, so that small batches still fill the chip in a single launch:
// kMidBlock threads while there are more rows than CUs, kWideBlock threads
// up to one row per CU, and G workgroups of kSplitBlock threads per row
// (merged by a second kernel) when a row per CU would leave most CUs idle.
constexpr int64_t kWideRows = PR_WIDE_ROWS;
constexpr int kWideBlock = PR_WIDE_BLOCK;
constexpr int kMidBlock = PR_MID_BLOCK;
constexpr int kSplitBlock = PR_SPLIT_BLOCK;
#ifndef PR_WIDE_TARGET
#define PR_WIDE_TARGET 256
#endif
constexpr int kWideTarget = PR_WIDE_TARGET;  // wide workgroups per launch: one per CU

int row_split(int64_t n_rows, int32_t V, pr_dtype dtype) {
  const int VEC = dtype == PR_BF16 ? 8 : 4;
  const int64_t nvec = V / VEC;
  if (n_rows <= 0 || n_rows >= kWideTarget) return 1;
  int64_t G = kWideTarget / n_rows;  // one round of at most kWideTarget workgroups
  const int64_t by_work = nvec / (kSplitBlock * 4);  // at least ~4 vectors per lane
  if (G > by_work) G = by_work;
  if (G > kMaxSplit) G = kMaxSplit;
  if (G < 1) G = 1;
  return static_cast<int>(G);
}

#ifndef PR_WIDE_LOAD_DEPTH_BF16
#define PR_WIDE_LOAD_DEPTH_BF16 2
#endif
#ifndef PR_WIDE_LOAD_DEPTH_F32
#define PR_WIDE_LOAD_DEPTH_F32 4
#endif

template <typename Tin>
static hipError_t launch_typed(const RowArgs& a, hipStream_t stream) {
  constexpr int U = unroll_for<Tin>();
  constexpr int LD = load_depth_for<Tin>();
  // Wide workgroups serve small batches, where each lane has few vectors; 16
  // waves per CU keep the loads in flight, so a shallow per-lane pipeline
  // (less padding in the last rounds) serves them best.
  constexpr int LDW = Elem<Tin>::kVec == 8 ? PR_WIDE_LOAD_DEPTH_BF16 : PR_WIDE_LOAD_DEPTH_F32;
  const dim3 grid(static_cast<unsigned>(a.n_rows * a.G));
  if (a.n_rows >= kWideRows) {
    row_features_kernel<Tin, kFeatBlock, U, LD, false><<<grid, kFeatBlock, 0, stream>>>(a);
  } else if (a.n_rows > 256) {
    row_features_kernel<Tin, kMidBlock, U, LDW, false><<<grid, kMidBlock, 0, stream>>>(a);
  } else if (a.G == 1) {
    row_features_kernel<Tin, kWideBlock, U, LDW, false><<<grid, kWideBlock, 0, stream>>>(a);
  } else {
    row_features_kernel<Tin, kSplitBlock, U, LDW, true><<<grid, kSplitBlock, 0, stream>>>(a);
    row_merge_kernel<<<dim3(static_cast<unsigned>(a.n_rows)), kWave, 0, stream>>>(a);
  }
  return hipGetLastError();
}

hipError_t launch_row_features(const RowArgs& a, pr_dtype dtype, hipStream_t stream) {
  if (a.n_rows == 0) return hipSuccess;
  return dtype == PR_BF16 ? launch_typed<uint16_t>(a, stream) : launch_typed<float>(a, stream);
}

// The sequence variant: the tiers of launch_typed, with one workgroup per row
// at every batch size.
template <typename Tin>
static hipError_t launch_sequence_typed(const RowArgs& a, hipStream_t stream) {
  constexpr int U = unroll_for<Tin>();
  constexpr int LD = load_depth_for<Tin>();
  constexpr int LDW = Elem<Tin>::kVec == 8 ? PR_WIDE_LOAD_DEPTH_BF16 : PR_WIDE_LOAD_DEPTH_F32;
  const dim3 grid(static_cast<unsigned>(a.n_rows));
  if (a.n_rows >= kWideRows) {
    row_features_kernel<Tin, kFeatBlock, U, LD, false, true><<<grid, kFeatBlock, 0, stream>>>(a);
  } else if (a.n_rows > 256) {
    row_features_kernel<Tin, kMidBlock, U, LDW, false, true><<<grid, kMidBlock, 0, stream>>>(a);
  } else {
    row_features_kernel<Tin, kWideBlock, U, LDW, false, true><<<grid, kWideBlock, 0, stream>>>(a);
  }
  return hipGetLastError();
}

hipError_t launch_feature_sequence(const RowArgs& a, pr_dtype dtype, hipStream_t stream) {
  if (a.n_rows == 0) return hipSuccess;
  return dtype == PR_BF16 ? launch_sequence_typed<uint16_t>(a, stream) : launch_sequence_typed<float>(a, stream);
}

// The sampling variant: the tiers of the sequence variant, with the
// sequence X when a.X is set.
// Float32 rows take two vectors per step and two loads in flight here (the
// other variants four and four): with the draw's state the float32 sampling
// kernels had spilled up to 163 registers.
template <typename Tin, bool SEQ>
static hipError_t launch_sample_typed(const RowArgs& a, hipStream_t stream) {
  constexpr bool kBf16 = Elem<Tin>::kVec == 8;
  constexpr int U = kBf16 ? unroll_for<Tin>() : 2;  // the same with and without X: the draw depends on U
  constexpr int LD = kBf16 ? load_depth_for<Tin>() : 2;
  constexpr int LDW = kBf16 ? PR_WIDE_LOAD_DEPTH_BF16 : 2;
  const dim3 grid(static_cast<unsigned>(a.n_rows));
  if (a.n_rows >= kWideRows) {
    row_features_kernel<Tin, kFeatBlock, U, LD, false, SEQ, true><<<grid, kFeatBlock, 0, stream>>>(a);
  } else if (a.n_rows > 256) {
    row_features_kernel<Tin, kMidBlock, U, LDW, false, SEQ, true><<<grid, kMidBlock, 0, stream>>>(a);
  } else {
    row_features_kernel<Tin, kWideBlock, U, LDW, false, SEQ, true><<<grid, kWideBlock, 0, stream>>>(a);
  }
  return hipGetLastError();
}

hipError_t launch_sample(const RowArgs& a, pr_dtype dtype, hipStream_t stream) {
  if (a.n_rows == 0) return hipSuccess;
  if (dtype == PR_BF16) return a.X ? launch_sample_typed<uint16_t, true>(a, stream)
                                   : launch_sample_typed<uint16_t, false>(a, stream);
  return a.X ? launch_sample_typed<float, true>(a, stream) : launch_sample_typed<float, false>(a, stream);
}

}  // namespace pr
